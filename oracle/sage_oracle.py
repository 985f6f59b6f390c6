"""CPU oracle for the scheduling-decision path (test infrastructure only).

Plain, slow, fp64 NumPy restatements of what each stage computes, written
from the paper's definitions. Only ``tests/``, ``__graft_entry__.smoke()``
and the ``cpu_baseline`` leg of ``bench.py`` may import this module; the
product path never does, and it imports nothing from the product package.

Stages and the passages they follow:

* ``round_to_bf16``   - storage of the history store / query batch: fp32
  embeddings rounded to bf16, round-to-nearest-even (a precision choice of
  this build; the paper does not fix one).
* ``similarity``      - Sec. 3.1: cosine similarity of prompt embeddings;
  for unit vectors that is the inner product (flat search, Sec. 3.1 footnote).
* ``topk``            - Sec. 3.1: the most similar history records, taken as
  the first ``k`` under (similarity desc, history index asc).
* ``histogram``       - Sec. 3.1: the neighbours' output lengths form the
  predicted distribution; records below the similarity threshold (0.8 by
  default) get no weight, the others weigh by their similarity, and the
  lengths are binned on log-spaced bins.
* ``cost``            - Sec. 3.2, unified cost model: C = O^2/2 + I*O.
* ``gittins``         - Sec. 3.3, Gittins index
  G(D) = inf_{Delta>0} E[min(X, Delta)] / P(X <= Delta), X ~ D.
* ``rank``            - Sec. 3.3: the smaller index is served first; ties go
  to the lower request id.
* ``length_similarity`` / ``predict_by_length`` - Sec. 4.3's semantic-unaware
  predictor: neighbours by similar input length instead of similar prompt.

Every function here is pinned by ``-m "not gpu"`` tests against brute force,
exact rational arithmetic, closed forms and invariants (tests/test_oracle_*.py).
"""
from __future__ import annotations

import os
from concurrent.futures import ThreadPoolExecutor

import numpy as np

NEG_INF = -np.inf


# ---------------------------------------------------------------- storage
def round_to_bf16(x) -> np.ndarray:
    """fp32 -> bf16 bit patterns (uint16), round to nearest, ties to even.

    A bf16 keeps the top 16 bits of an fp32. Rounding adds half of the
    dropped range (0x7FFF) plus the kept part's lowest bit, so that an exact
    half-way case rounds to the even neighbour. Inputs must be finite.
    """
    x = np.ascontiguousarray(x, dtype=np.float32)
    if not np.all(np.isfinite(x)):
        raise ValueError("round_to_bf16: non-finite input")
    u = x.view(np.uint32).astype(np.uint64)
    keep_lsb = (u >> np.uint64(16)) & np.uint64(1)
    r = (u + np.uint64(0x7FFF) + keep_lsb) >> np.uint64(16)
    return r.astype(np.uint16)


def bf16_to_f64(bits) -> np.ndarray:
    """Exact value of bf16 bit patterns as fp64."""
    b = np.ascontiguousarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)
    return b.view(np.float32).astype(np.float64)


# ------------------------------------------------------------- similarity
def store_insert(ring_bits, ring_len, total: int, emb_f32, out_len, capacity: int):
    """FIFO history window (Sec. 3.1): record t of all records ever inserted
    (counting from 0) is kept in row t mod capacity, so each new record
    replaces the oldest once the window is full. Inserts a batch in order and
    returns the updated (ring_bits, ring_len, total)."""
    bits = np.array(ring_bits, dtype=np.uint16, copy=True)
    lens = np.array(ring_len, dtype=np.int32, copy=True)
    new_bits = round_to_bf16(np.asarray(emb_f32, dtype=np.float32))
    for i in range(new_bits.shape[0]):
        slot = (int(total) + i) % capacity
        bits[slot] = new_bits[i]
        lens[slot] = int(out_len[i])
    return bits, lens, int(total) + new_bits.shape[0]


def similarity(q_bits, h_bits) -> np.ndarray:
    """s[q, n] = sum_t Q[q, t] * H[n, t] over the stored bf16 values, in fp64.

    Products of two bf16 values are exact in fp64; the sums are exact or
    within a few fp64 ulps for the dimensions used here. No renormalisation
    after the bf16 rounding. Either operand may be given as bf16 bit
    patterns (uint16) or as their exact fp64 values (``bf16_to_f64``), so
    that a large store is widened once for several query blocks.
    """
    widen = lambda a: a if np.asarray(a).dtype == np.float64 else bf16_to_f64(a)
    return widen(q_bits) @ widen(h_bits).T


# ------------------------------------------------------------------ top-k
def topk_row(s: np.ndarray, k: int):
    """First ``k`` history indices under (s desc, n asc), padded with (-1, -inf).

    All indices whose score reaches the m-th largest value (m = min(k, N))
    are kept before the lexicographic sort, so ties at the boundary are
    resolved by the index rule, never by the selection routine.
    """
    N = s.shape[0]
    m = min(k, N)
    if m < N:
        t = -np.partition(-s, m - 1)[m - 1]
        cand = np.nonzero(s >= t)[0]
    else:
        cand = np.arange(N)
    order = cand[np.lexsort((cand, -s[cand]))][:m]
    ids = np.full(k, -1, dtype=np.int32)
    sims = np.full(k, NEG_INF, dtype=np.float64)
    ids[:m] = order
    sims[:m] = s[order]
    return ids, sims


def topk(S: np.ndarray, k: int):
    Q = S.shape[0]
    ids = np.empty((Q, k), dtype=np.int32)
    sims = np.empty((Q, k), dtype=np.float64)
    for q in range(Q):
        ids[q], sims[q] = topk_row(S[q], k)
    return ids, sims


def search(q_bits, h_bits, k: int, block: int = 128, threads: int | None = None):
    """Similarity + top-k over the whole store, one query block at a time.

    Blocking over queries only bounds memory; each row is still the plain
    definition (full fp64 score row, then ``topk_row``). The store may be
    given already widened to fp64 (``bf16_to_f64``).
    """
    Q = q_bits.shape[0]
    hf = h_bits if np.asarray(h_bits).dtype == np.float64 else bf16_to_f64(h_bits)
    ids = np.empty((Q, k), dtype=np.int32)
    sims = np.empty((Q, k), dtype=np.float64)
    threads = threads or os.cpu_count() or 1
    with ThreadPoolExecutor(max_workers=threads) as pool:
        for s0 in range(0, Q, block):
            e0 = min(Q, s0 + block)
            S = bf16_to_f64(q_bits[s0:e0]) @ hf.T
            rows = list(pool.map(lambda r: topk_row(S[r], k), range(e0 - s0)))
            for r, (i, v) in enumerate(rows):
                ids[s0 + r], sims[s0 + r] = i, v
    return ids, sims


def length_similarity(prompt_len, hist_prompt_len, max_len: int) -> np.ndarray:
    """Input-length similarity of the semantic-unaware predictor (Sec. 4.3's
    predictor ablation: history records with a similar input length stand in
    for similar prompts). Reading: s(I, L) = min(I, L) / max(I, L), the
    ratio of the shorter to the longer prompt, in (0, 1] and 1 for equal
    lengths, so that the predictor's similarity threshold (0.8) keeps its
    meaning (within a factor 1.25). It is defined as the fp32 quotient of the
    two lengths (correctly rounded), the precision in which the neighbour
    choice is made. Lengths below 1 count as 1, history lengths above
    max_len as max_len. Returns [Q, N] fp32 values widened to fp64."""
    I = np.maximum(np.asarray(prompt_len, dtype=np.int64), 1)[:, None]
    L = np.clip(np.asarray(hist_prompt_len, dtype=np.int64), 1, int(max_len))[None, :]
    a = np.minimum(I, L).astype(np.float32)
    b = np.maximum(I, L).astype(np.float32)
    return (a / b).astype(np.float64)


# -------------------------------------------------------------- histogram
def bin_of(lengths, edges) -> np.ndarray:
    """Largest b in [0, B-1] with edges[b] <= L (lengths below edges[0] -> 0)."""
    B = edges.shape[0] - 1
    b = np.searchsorted(edges, np.asarray(lengths, dtype=np.float64), side="right") - 1
    return np.clip(b, 0, B - 1).astype(np.int64)


def histogram(ids, sims, hist_len, edges, tau: float, weighting: str = "similarity"):
    """Per-request output-length distribution from its neighbours.

    counts[q, b]: neighbours (valid ids only) whose length falls in bin b.
    mass[q, b]  : sum of w_i over those neighbours / sum of all w_i, where
                  w_i = s_i if s_i >= tau else 0; if every w_i is 0 the mass
                  falls back to counts / (number of valid neighbours).
    weighting="uniform" is the paper's own form (Sec. 3.1): every neighbour
    at or above the threshold counts once, w_i = 1 if s_i >= tau else 0.
    """
    if weighting not in ("similarity", "uniform"):
        raise ValueError(f"histogram: unknown weighting {weighting!r}")
    ids = np.asarray(ids)
    sims = np.asarray(sims, dtype=np.float64)
    Q, _ = ids.shape
    B = edges.shape[0] - 1
    counts = np.zeros((Q, B), dtype=np.int32)
    mass = np.zeros((Q, B), dtype=np.float64)
    tau = float(np.float32(tau))
    for q in range(Q):
        valid = ids[q] >= 0
        m = int(valid.sum())
        if m == 0:
            continue
        b = bin_of(hist_len[ids[q][valid]], edges)
        s = sims[q][valid]
        w = np.where(s >= tau, s if weighting == "similarity" else 1.0, 0.0)
        np.add.at(counts[q], b, 1)
        W = w.sum()
        if W > 0:
            np.add.at(mass[q], b, w)
            mass[q] /= W
        else:
            mass[q] = counts[q] / m
    return counts, mass


# ------------------------------------------------------------------- cost
def cost(prompt_len, bin_repr) -> np.ndarray:
    """Service cost of each support point: x[q, b] = r_b^2 / 2 + I_q * r_b."""
    I = np.asarray(prompt_len, dtype=np.float64)[:, None]
    r = np.asarray(bin_repr, dtype=np.float64)[None, :]
    return r * r / 2.0 + I * r


def cost_variant(prompt_len, bin_repr, model: str) -> np.ndarray:
    """The cost models the paper compares against (Sec. 4 ablation):
    "resource" = O^2/2 + I O (the adopted one, ``cost``), "output" = O (the
    output length alone), "overall" = I + 2 O (input and output lengths,
    output weighted double), each at O = r_b."""
    I = np.asarray(prompt_len, dtype=np.float64)[:, None]
    r = np.asarray(bin_repr, dtype=np.float64)[None, :]
    if model == "resource":
        return cost(prompt_len, bin_repr)
    if model == "output":
        return np.broadcast_to(r, (I.shape[0], r.shape[1])).copy()
    if model == "overall":
        return I + 2.0 * r
    raise ValueError(f"cost_variant: unknown model {model!r}")


def mix_uniform(mass, weight: float) -> np.ndarray:
    """A prediction made deliberately inaccurate (Sec. 4 ablation): a uniform
    distribution over the bins merged with the row's distribution at
    weight : (1 - weight), i.e. 1:4 for weight 0.2. Rows with no mass stay
    empty."""
    p = np.asarray(mass, dtype=np.float64)
    B = p.shape[1]
    tot = p.sum(axis=1, keepdims=True)
    with np.errstate(divide="ignore", invalid="ignore"):
        mixed = (1.0 - weight) * p / tot + weight / B
    return np.where(tot > 0, mixed, p)


def mean_index(mass, x):
    """The Mean baseline (Sec. 4 ablation): E[X] = sum p x / sum p; +inf for
    a row with no mass."""
    p = np.asarray(mass, dtype=np.float64)
    x = np.asarray(x, dtype=np.float64)
    if x.ndim == 1:
        x = np.broadcast_to(x, p.shape)
    tot = p.sum(axis=1)
    with np.errstate(divide="ignore", invalid="ignore"):
        return np.where(tot > 0, (p * x).sum(axis=1) / tot, np.inf)


# ----------------------------------------------------------------- index
def gittins(mass, x):
    """Gittins index of each row's discrete cost distribution.

    With support points x_0 <= x_1 <= ... (non-decreasing, as the cost is
    increasing in the output length) and masses p_b:
        F_b = sum_{j<=b} p_j,  S_b = sum_{j<=b} p_j x_j,  T_b = sum_{j>b} p_j,
        G   = min over b with F_b > 0 of (S_b + T_b x_b) / F_b.
    For Delta in [x_b, x_{b+1}) the completion probability is F_b and the
    expected spend S_b + T_b Delta grows with Delta, so the infimum over
    Delta is reached at a support point. Rows with no mass get +inf (and
    argmin -1). The index does not depend on the scale of p, so rows need
    not sum to one. Returns (G, argmin) with argmin the smallest b at the min.
    """
    p = np.asarray(mass, dtype=np.float64)
    x = np.asarray(x, dtype=np.float64)
    if x.ndim == 1:
        x = np.broadcast_to(x, p.shape)
    if np.any(np.diff(x, axis=1) < 0):
        raise ValueError("gittins: support must be non-decreasing along each row")
    F = np.cumsum(p, axis=1)
    S = np.cumsum(p * x, axis=1)
    tail = np.cumsum(p[:, ::-1], axis=1)[:, ::-1]         # sum over j >= b
    T = np.zeros_like(p)
    T[:, :-1] = tail[:, 1:]                               # sum over j > b
    with np.errstate(divide="ignore", invalid="ignore"):
        ratio = np.where(F > 0, (S + T * x) / F, np.inf)
    G = ratio.min(axis=1)
    arg = np.where(np.isfinite(G), ratio.argmin(axis=1), -1).astype(np.int32)
    return G, arg


def attained_service(prompt_len, generated, bucket: int) -> np.ndarray:
    """Service already received by a running request, at its last refresh.

    Sec. 3.3 refreshes a running request's index only at bucket boundaries
    (bucket size 200 by default, Sec. 4); reading: a boundary every `bucket`
    generated tokens. The service is the cost model of Sec. 3.2 at the
    boundary: o = bucket * floor(generated / bucket), a = o^2 / 2 + I * o.
    """
    if bucket < 1:
        raise ValueError("attained_service: bucket must be >= 1")
    I = np.asarray(prompt_len, dtype=np.float64)
    o = np.floor(np.asarray(generated, dtype=np.float64) / bucket) * bucket
    return o * o / 2.0 + I * o


def gittins_attained(mass, x, a):
    """Gittins index of the remaining cost of running requests (Sec. 3.3).

    A request that has received service a is known to need X > a, and what
    remains is Y = X - a. Its index is the Gittins index of Y:
        inf over Delta > 0 of E[min(X - a, Delta); X > a] / P(a < X <= a + Delta),
    i.e. ``gittins`` applied to the masses of the support points above a
    (those at or below a are ruled out) shifted down by a. a = 0 gives the
    index at arrival. A row with no mass above a gets +inf (argmin -1).
    """
    p = np.asarray(mass, dtype=np.float64)
    x = np.asarray(x, dtype=np.float64)
    if x.ndim == 1:
        x = np.broadcast_to(x, p.shape)
    a = np.asarray(a, dtype=np.float64).reshape(-1, 1)
    alive = x > a
    return gittins(np.where(alive, p, 0.0), np.where(alive, x - a, 0.0))


# ------------------------------------------------------------------ rank
def rank(G) -> np.ndarray:
    """Queue order: ascending index, ties to the lower request id."""
    return np.argsort(np.asarray(G), kind="stable").astype(np.int32)


# -------------------------------------------------------------- pipelines
def predict(queries_f32, hist_f32, hist_len, k, tau, edges, *, block=128, threads=None):
    """Stages storage -> similarity -> top-k -> histogram for a query batch."""
    qb = round_to_bf16(queries_f32)
    hb = round_to_bf16(hist_f32)
    ids, sims = search(qb, hb, k, block=block, threads=threads)
    counts, mass = histogram(ids, sims, hist_len, edges, tau)
    return ids, sims, counts, mass


def predict_by_length(prompt_len, hist_prompt_len, max_len, hist_len, k, tau, edges):
    """The semantic-unaware history-based predictor (Sec. 4.3): the k history
    records with the most similar input length (``length_similarity``, ties
    to the lower index), then the same similarity-weighted histogram as the
    semantic predictor ("the same filtering method")."""
    S = length_similarity(prompt_len, hist_prompt_len, max_len)
    ids, sims = topk(S, k)
    counts, mass = histogram(ids, sims, hist_len, edges, tau)
    return ids, sims, counts, mass


def schedule(mass, prompt_len, bin_repr):
    """Stages cost -> index -> rank."""
    x = cost(prompt_len, bin_repr)
    G, arg = gittins(mass, x)
    return G, arg, rank(G)
