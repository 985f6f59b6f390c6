"""Pins of the semantic-unaware (input-length) predictor of the oracle
(Sec. 4.3's predictor ablation)."""
import os
from fractions import Fraction

import numpy as np
import pytest

import oracle
from paper_2603_07917_amd import workloads

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _golden():
    kv = {}
    for line in open(os.path.join(GOLDEN, "length_neighbours.txt")):
        if line.startswith("#") or not line.strip():
            continue
        key, val = line.split(":", 1)
        kv[key.strip()] = val.strip()
    return kv


def test_length_neighbours_golden():
    kv = _golden()
    I = np.array([int(kv["query_len"])])
    L = np.array([int(v) for v in kv["hist_prompt_len"].split()])
    S = oracle.length_similarity(I, L, 1000)
    k = int(kv["k"])
    ids, sims = oracle.topk(S, len(L))
    assert list(ids[0]) == [int(v) for v in kv["order"].split()]
    ids, sims = oracle.topk(S, k)
    assert list(ids[0]) == [int(v) for v in kv["neighbours"].split()]
    want = [float(np.float32(float(Fraction(v)))) for v in kv["sims"].split()]
    assert list(sims[0]) == want


def _exact_order(I, L):
    """Brute force: history indices by the exact rational min/max desc, ties by index."""
    keys = []
    for n, l in enumerate(L):
        a, b = min(max(I, 1), max(l, 1)), max(max(I, 1), max(l, 1))
        keys.append((-Fraction(a, b), n))
    return [n for _, n in sorted(keys)]


@pytest.mark.parametrize("seed", range(5))
def test_length_neighbours_match_exact_rationals(seed):
    # lengths <= 1000: distinct ratios differ by >= 1e-6, far above the fp32
    # rounding of a quotient near 1 (6e-8), so the fp32 order is the exact one
    rng = np.random.default_rng(seed)
    L = rng.integers(1, 1001, size=300)
    L[:40] = L[40:80]                                   # repeated lengths: ties by index
    Iq = rng.integers(1, 1001, size=12)
    Iq[0] = L[7]                                        # a query whose length is in the store
    S = oracle.length_similarity(Iq, L, 1000)
    for q in range(len(Iq)):
        ids, _ = oracle.topk(S[q:q + 1], 37)
        assert list(ids[0]) == _exact_order(int(Iq[q]), L)[:37]


def test_length_similarity_properties():
    L = np.array([1, 5, 10, 20, 40, 5000, 7000])
    S = oracle.length_similarity(np.array([10, 0, 9000]), L, 6000)
    assert S[0, 2] == 1.0 and S[0, 1] == S[0, 3] == 0.5          # symmetric in the ratio
    assert np.all((S > 0) & (S <= 1))
    assert S[1, 0] == 1.0                                          # lengths below 1 count as 1
    assert S[2, 6] == np.float32(6000) / np.float32(9000)                # clamped to max_len
    assert S[2, 5] == np.float32(5000) / np.float32(9000)
    # the full predictor: the same histogram as the semantic one
    edges, _ = workloads.log_bins(1000, 8)
    out = np.arange(1, 8) * 100
    ids, sims, counts, mass = oracle.predict_by_length(np.array([10]), L, 6000, out, 3, 0.8, edges)
    assert list(ids[0]) == [2, 1, 3] and counts[0].sum() == 3
    assert np.isclose(mass[0].sum(), 1.0)                           # no weight reaches 0.8 but one
    b = oracle.bin_of([300], edges)[0]
    assert mass[0, b] == 1.0                                        # only record 2 (s = 1) weighs
