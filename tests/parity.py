"""Parity checks between the HIP path's outputs and the oracle's.

The oracle only ever sees the seeded inputs: it computes its own neighbours,
histograms, indices and orders, and the GPU's results are compared against
those. Nothing the GPU produced is fed to the oracle.

Tolerances (fixed by the path's precision):

* similarities within 1e-4 absolute (fp32 accumulation of bf16 products);
* neighbour sets exact except for items within 1e-4 of the k-th score;
* counts bit-exact on the same neighbour set; masses within a bound derived
  from the row's measured similarity error (``mass_bound``);
* on the same inputs, cost and index within 1e-5 relative; downstream of
  predict, the index inside the interval that the mass bound allows
  (``index_interval``), widened by the same 1e-5;
* rank bit-exact against a stable argsort of the same (generated) keys;
  downstream of the index, the order is a stable ascending sort of the
  GPU's own index values (a property, checked without the oracle).
"""
from __future__ import annotations

import numpy as np

import oracle

SIM_TOL = 1e-4
MASS_TOL = 1e-6          # masses on identical neighbour inputs (stage tests)
INDEX_RTOL = 1e-5
U32 = 2.0 ** -24         # fp32 unit roundoff


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
        assert err.max(initial=0.0) <= tol, f"sim error {err.max()} at query {q}"
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


def mass_bound(n_weighted: int, W: float, e: float, k: int) -> float:
    """Largest |mass'_b - mass_b| (and L1 distance) when each of the n weighted
    neighbours' similarity moves by at most e: with W = sum of the weights,
    |dW_b| <= n_b e and |dW| <= n e, so sum_b |d(W_b / W)| <= 2 n e / (W - n e);
    plus the fp32 rounding of a k-term sum and a division."""
    fp = (k + 4) * U32
    if n_weighted == 0 or W <= 0:
        return fp
    return 2.0 * n_weighted * e / (W - n_weighted * e) + fp


def check_predict(gids, gsims, gcounts, gmass, S, hist_len, edges, tau, k, min_clean=0.5):
    """GPU predict outputs against the oracle's own prediction from the scores S.

    Neighbours as ``check_topk``. A row is clean when the GPU chose the
    oracle's neighbour set and no neighbour's score lies within the row's
    similarity error of tau (so every weight decision is the same). On clean
    rows the counts are bit-exact and the masses within ``mass_bound``.
    Returns (clean [Q] bool, oracle mass [Q, B] fp64, L1 bound [Q]).
    """
    Q = S.shape[0]
    check_topk(gids, gsims, S, k)
    ids_o, sims_o = oracle.topk(S, k)
    counts_o, mass_o = oracle.histogram(ids_o, sims_o, hist_len, edges, tau)
    t32 = float(np.float32(tau))
    clean = np.zeros(Q, dtype=bool)
    delta = np.full(Q, np.inf)
    for q in range(Q):
        v = gids[q][gids[q] >= 0].astype(np.int64)
        vo = ids_o[q][ids_o[q] >= 0]
        if set(v.tolist()) != set(vo.tolist()):
            continue
        e = max(float(np.abs(gsims[q][:len(v)].astype(np.float64) - S[q, v]).max(initial=0.0)), U32)
        s = S[q, vo]
        if np.any(np.abs(s - t32) <= e):
            continue
        clean[q] = True
        w = np.where(s >= t32, s, 0.0)
        delta[q] = mass_bound(int((w > 0).sum()), float(w.sum()), e, k)
        assert np.array_equal(gcounts[q], counts_o[q]), f"counts differ, query {q}"
        err = np.abs(gmass[q].astype(np.float64) - mass_o[q])
        assert err.max() <= delta[q], f"mass error {err.max()} > {delta[q]}, query {q}"
    assert clean.mean() >= min_clean, f"only {clean.sum()} of {Q} rows comparable"
    return clean, mass_o, delta


def check_hist(gids, gsims, gcounts, gmass, hist_len, edges, tau):
    """Histogram stage on generated neighbour lists (the same inputs on both
    sides): counts bit-exact, masses within MASS_TOL."""
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


def index_interval(mass, x, delta):
    """[lo, hi] holding the Gittins index of every distribution within L1
    distance delta of each row of `mass`.

    With N_b = sum_j p_j min(x_j, x_b) and F_b = sum_{j<=b} p_j the index is
    min_b N_b / F_b. A change of L1 size delta moves N_b by at most x_b delta
    and F_b by at most delta, so every ratio lies in
    [(N_b - x_b delta) / (F_b + delta), (N_b + x_b delta) / (F_b - delta)].
    """
    p = np.asarray(mass, dtype=np.float64)
    x = np.broadcast_to(np.asarray(x, dtype=np.float64), p.shape)
    F = np.cumsum(p, axis=1)
    S = np.cumsum(p * x, axis=1)
    tail = np.cumsum(p[:, ::-1], axis=1)[:, ::-1]
    T = np.zeros_like(p)
    T[:, :-1] = tail[:, 1:]
    Nb = S + T * x
    d = np.asarray(delta, dtype=np.float64)[:, None]
    with np.errstate(divide="ignore", invalid="ignore"):
        lo = np.where(F + d > 0, np.maximum(Nb - x * d, 0.0) / (F + d), np.inf).min(axis=1)
        hi = np.where(F > d, (Nb + x * d) / (F - d), np.inf).min(axis=1)
    return lo, hi


def check_index_downstream(g_gpu, mass_o, x, delta, rows):
    """GPU index of predicted rows inside the interval the mass bound allows."""
    lo, hi = index_interval(mass_o[rows], x[rows] if np.ndim(x) == 2 else x, delta[rows])
    g = g_gpu[rows].astype(np.float64)
    assert np.all(np.isfinite(g) & np.isfinite(hi)), "non-finite index on a predicted row"
    bad = (g < lo * (1 - INDEX_RTOL)) | (g > hi * (1 + INDEX_RTOL))
    assert not bad.any(), f"index outside its interval on {int(bad.sum())} rows"
    return lo, hi


def check_rank(order, g):
    """Bit-exact against a stable ascending argsort of the same (generated) keys."""
    want = oracle.rank(g)
    assert np.array_equal(order, want), "rank differs from the stable argsort"


def check_sorted_stably(order, g):
    """Property of a rank output: a permutation that puts its own keys in
    ascending order, equal keys by ascending id."""
    n = len(g)
    assert order.shape == (n,) and np.array_equal(np.sort(order), np.arange(n)), "not a permutation"
    v = np.asarray(g)[order]
    ok = (v[:-1] < v[1:]) | ((v[:-1] == v[1:]) & (order[:-1] < order[1:]))
    assert np.all(ok), "order is not a stable ascending sort of its keys"


def check_rank_vs_oracle(order, G_o, rtol=INDEX_RTOL):
    """A rank output against the oracle's index values G_o of the same rows:
    two requests may come out of the oracle's order only when their values
    are within rtol relative of each other, i.e. along the GPU's order every
    value is at least the largest one before it, shrunk by rtol (+inf rows
    last)."""
    v = np.asarray(G_o, dtype=np.float64)[np.asarray(order)]
    fin = np.isfinite(v)
    n_fin = int(fin.sum())
    assert np.all(fin[:n_fin]) and not np.any(fin[n_fin:]), "+inf rows are not last"
    run = np.maximum.accumulate(v[:n_fin])
    bad = v[:n_fin] < run * (1.0 - rtol) - 1e-300
    assert not bad.any(), f"order departs from the oracle's beyond {rtol} relative at {np.nonzero(bad)[0][:5]}"
