"""Parity checks between the HIP path's outputs and the oracle's.

Tolerances (fixed by the path's precision): similarities within 1e-4
absolute (fp32 accumulation of bf16 products); neighbour sets exact except
for items within 1e-4 of the k-th score; counts bit-exact on the same
neighbours; masses within 1e-6 absolute; cost and index within 1e-5 relative.
"""
from __future__ import annotations

import numpy as np

import oracle

SIM_TOL = 1e-4
MASS_TOL = 1e-6
INDEX_RTOL = 1e-5


def check_topk(gids: np.ndarray, gsims: np.ndarray, S: np.ndarray, k: int, tol: float = SIM_TOL):
    """GPU neighbours of some queries against the oracle's fp64 score rows S.

    * every returned similarity is within tol of the oracle's score of that id;
    * every id scoring above s_k + tol is returned, none below s_k - tol
      (s_k: the oracle's k-th score); items in the band may differ;
    * the list is sorted by the GPU's own fp32 scores, ties by lower id;
    * padding (-1, -inf) exactly when N < k.
    Returns the number of queries whose id set equals the oracle's.
    """
    Qs, N = S.shape
    m = min(k, N)
    equal = 0
    for q in range(Qs):
        ids, sims = gids[q], gsims[q]
        assert np.all(ids[m:] == -1) and np.all(np.isneginf(sims[m:])), f"padding, query {q}"
        v = ids[:m].astype(np.int64)
        assert np.all((v >= 0) & (v < N)), f"id range, query {q}"
        assert len(np.unique(v)) == m, f"duplicate ids, query {q}"
        err = np.abs(sims[:m].astype(np.float64) - S[q, v])
        assert err.max() <= tol, f"sim error {err.max()} at query {q}"
        s32 = sims[:m]
        ok = (s32[:-1] > s32[1:]) | ((s32[:-1] == s32[1:]) & (v[:-1] < v[1:]))
        assert np.all(ok), f"order, query {q}"
        sk = -np.partition(-S[q], m - 1)[m - 1]
        must = np.nonzero(S[q] > sk + tol)[0]
        assert np.isin(must, v).all(), f"missing a neighbour above the band, query {q}"
        assert np.all(S[q, v] >= sk - tol), f"neighbour below the band, query {q}"
        want, _ = oracle.topk_row(S[q], k)
        if set(want[:m].tolist()) == set(v.tolist()):
            equal += 1
            # positions agree except for swaps of items whose oracle scores are within tol
            for i in np.nonzero(want[:m] != v)[0]:
                assert abs(S[q, want[i]] - S[q, v[i]]) <= tol, f"position {i}, query {q}"
    return equal


def check_hist(gids, gsims, gcounts, gmass, hist_len, edges, tau):
    """Counts bit-exact and masses within MASS_TOL of the oracle on the GPU's neighbours."""
    c, m = oracle.histogram(gids, gsims.astype(np.float64), hist_len, edges, tau)
    assert np.array_equal(gcounts, c), "counts differ"
    err = np.abs(gmass.astype(np.float64) - m)
    assert err.max() <= MASS_TOL, f"mass error {err.max()}"
    valid = (gids >= 0).sum(1)
    assert np.array_equal(gcounts.sum(1), valid)
    tot = gmass.astype(np.float64).sum(1)
    assert np.all(np.abs(tot[valid > 0] - 1.0) <= MASS_TOL * 4)
    assert np.all(tot[valid == 0] == 0.0)


def check_index(g_gpu, mass, x):
    """Index within INDEX_RTOL relative of the oracle's on the same masses; +inf matches +inf."""
    G, _ = oracle.gittins(mass.astype(np.float64), x)
    inf = np.isinf(G)
    assert np.array_equal(np.isinf(g_gpu), inf), "+inf rows differ"
    rel = np.abs(g_gpu[~inf].astype(np.float64) - G[~inf]) / np.abs(G[~inf])
    assert rel.max(initial=0.0) <= INDEX_RTOL, f"index relative error {rel.max()}"
    return G


def check_rank(order, g):
    """Bit-exact against a stable ascending argsort of the same keys."""
    want = oracle.rank(g)
    assert np.array_equal(order, want), "rank differs from the stable argsort"
