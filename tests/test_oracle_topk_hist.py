"""Pins of the oracle's top-k and histogram stages (CPU only)."""
import os
from fractions import Fraction

import numpy as np
import pytest

import oracle
from paper_2603_07917_amd import workloads
from tests import brute

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


@pytest.mark.parametrize("seed", range(12))
def test_topk_equals_full_sort(seed):
    rng = np.random.default_rng(seed)
    N = int(rng.integers(1, 300))
    k = int(rng.integers(1, 70))
    # quantised scores force many exact ties, including at the k-th position
    s = np.round(rng.standard_normal(N) * 4) / 4
    ids, sims = oracle.topk_row(s, k)
    want = brute.topk_sorted(list(s), k)
    m = min(k, N)
    assert list(ids[:m]) == want
    assert np.all(ids[m:] == -1) and np.all(np.isneginf(sims[m:]))
    assert np.array_equal(sims[:m], s[want])


def test_topk_duplicates_lower_id_wins():
    s = np.array([0.5, 0.9, 0.9, 0.1, 0.9, 0.7])
    ids, _ = oracle.topk_row(s, 3)
    assert list(ids) == [1, 2, 4]
    ids, _ = oracle.topk_row(s, 2)
    assert list(ids) == [1, 2]


def test_topk_k_at_least_n_returns_all_and_pads():
    s = np.array([0.2, -0.4, 0.9])
    ids, sims = oracle.topk_row(s, 5)
    assert list(ids) == [2, 0, 1, -1, -1]
    assert sims[3] == -np.inf and sims[4] == -np.inf


def test_bin_of_every_integer_has_one_bin():
    for L_max, B in [(4096, 128), (8192, 256), (32768, 1024), (16, 4), (100, 7)]:
        edges, _ = workloads.log_bins(L_max, B)
        Ls = np.arange(1, L_max + 1)
        b = oracle.bin_of(Ls, edges)
        assert b.min() >= 0 and b.max() <= B - 1
        assert np.all(np.diff(b) >= 0)
        for L in sorted(set(range(1, min(40, L_max) + 1)) | set(range(max(1, L_max - 40), L_max + 1))):
            assert b[L - 1] == brute.bin_linear(L, list(edges))
        assert b[-1] == B - 1


def _golden_hist():
    g = {}
    for line in open(os.path.join(GOLDEN, "histogram_case.txt")):
        if line.startswith("#") or not line.strip():
            continue
        key, val = line.split(":", 1)
        g[key.strip()] = val.split()
    return g


def test_histogram_golden_case():
    g = _golden_hist()
    edges = np.array([float(v) for v in g["edges"]])
    ids = np.array([[int(v) for v in g["ids"]]], dtype=np.int32)
    sims = np.array([[float(v) for v in g["sims"]]])
    lengths = np.array([int(v) for v in g["lengths"]], dtype=np.int32)
    counts, mass = oracle.histogram(ids, sims, lengths, edges, float(g["tau"][0]))
    assert list(counts[0]) == [int(v) for v in g["counts"]]
    assert [Fraction(v).limit_denominator(1000) for v in mass[0]] == [Fraction(v) for v in g["mass"]]
    counts, mass = oracle.histogram(ids, sims, lengths, edges, float(g["fallback_tau"][0]))
    assert [Fraction(v).limit_denominator(1000) for v in mass[0]] == \
        [Fraction(v) for v in g["fallback_mass"]]


@pytest.mark.parametrize("seed", range(8))
def test_histogram_equals_exact_fractions(seed):
    rng = np.random.default_rng(100 + seed)
    N, k, B, L_max = 50, int(rng.integers(1, 20)), int(rng.integers(1, 12)), 300
    edges, _ = workloads.log_bins(L_max, B)
    lengths = rng.integers(1, L_max + 1, size=N).astype(np.int32)
    Q = 6
    ids = np.full((Q, k), -1, np.int32)
    sims = np.full((Q, k), -np.inf)
    for q in range(Q):
        m = int(rng.integers(1, k + 1))
        ids[q, :m] = rng.choice(N, size=m, replace=False)
        sims[q, :m] = np.sort(rng.uniform(0.5, 1.0, size=m).astype(np.float32))[::-1]
    tau = 0.8 if seed % 2 == 0 else 0.999
    counts, mass = oracle.histogram(ids, sims, lengths, edges, tau)
    for q in range(Q):
        c, m_ = brute.histogram_exact(list(ids[q]), list(sims[q]), list(lengths),
                                      list(edges), float(np.float32(tau)))
        assert list(counts[q]) == c
        assert np.allclose(mass[q], [float(v) for v in m_], rtol=0, atol=1e-15)
        assert counts[q].sum() == (ids[q] >= 0).sum()
        assert abs(mass[q].sum() - 1.0) < 1e-12


def test_histogram_single_length_single_bin():
    edges, _ = workloads.log_bins(4096, 128)
    ids = np.arange(32, dtype=np.int32)[None, :]
    sims = np.linspace(0.99, 0.81, 32)[None, :]
    lengths = np.full(32, 777, np.int32)
    counts, mass = oracle.histogram(ids, sims, lengths, edges, 0.8)
    b = brute.bin_linear(777, list(edges))
    assert counts[0, b] == 32 and counts[0].sum() == 32
    assert abs(mass[0, b] - 1.0) < 1e-15 and abs(mass[0].sum() - 1.0) < 1e-15


def test_histogram_threshold_above_all_is_count_fraction():
    rng = np.random.default_rng(7)
    edges, _ = workloads.log_bins(4096, 64)
    lengths = rng.integers(1, 4097, size=100).astype(np.int32)
    ids = rng.choice(100, size=(4, 20), replace=True).astype(np.int32)
    sims = rng.uniform(0.1, 0.7, size=(4, 20))
    counts, mass = oracle.histogram(ids, sims, lengths, edges, 0.8)
    assert np.allclose(mass, counts / 20.0, rtol=0, atol=0)


def test_predict_pipeline_on_generated_mixture():
    w = workloads.small_predict(Q=20, N=600, d=64, k=8, B=16, seed=3, clusters=4)
    ids, sims, counts, mass = oracle.predict(w.queries, w.hist_emb, w.hist_len, 8, 0.8,
                                             w.bin_edges)
    S = oracle.similarity(oracle.round_to_bf16(w.queries), oracle.round_to_bf16(w.hist_emb))
    for q in range(20):
        assert list(ids[q]) == brute.topk_sorted(list(S[q]), 8)
    # neighbours come from the query's own cluster (the mixture is well separated)
    assert np.mean(w.hist_cluster[ids] == w.query_cluster[:, None]) > 0.95
    assert np.all(counts.sum(1) == 8)
    assert np.allclose(mass.sum(1), 1.0, atol=1e-12)
