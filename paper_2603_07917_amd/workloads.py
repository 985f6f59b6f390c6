"""Seeded synthetic workloads for the scheduling-decision path.

This module draws inputs only: embeddings, recorded output lengths, prompt
lengths, bin edges and (for the index-only workload) length distributions.
It holds none of the method's arithmetic (no similarity, selection,
histogram, cost, index or ranking), so both the HIP path and the CPU oracle
may consume what it produces.

The paper evaluates on conversation / summarisation / document-writing
datasets that are not available here; these mixtures stand in for them
(Sec. 4.1 names the datasets; Sec. 3.1 motivates clustered prompts whose
similar members have similar output lengths).

Recipe (one ``numpy.random.Generator`` per purpose, spawned in a fixed order
from ``SeedSequence([260307917, config_id])``):

* cluster centres ``c_j ~ N(0, I_d)``, normalised;
* a point of cluster ``j`` is ``normalise(c_j + (sigma/sqrt(d)) g)`` with
  ``g ~ N(0, I_d)``, so the noise has RMS norm ``sigma`` (0.3 by default);
  ``noise_frac`` of the rows are instead uniform on the sphere;
* each cluster has a lognormal output-length law ``(mu_j, s_j)`` drawn
  uniformly from the configured ranges; a row's length is
  ``clamp(rint(exp(mu_j + s_j z)), 1, L_max)`` (noise rows borrow a
  uniformly chosen cluster's law);
* embeddings are produced in fp32 (unit norm up to fp32 rounding); rounding
  them to bf16 is a step of the path, not of this generator;
* log-spaced bins over ``[1, L_max]``: ``edges[b] = L_max ** (b / B)`` and
  representative lengths ``r_b = sqrt(edges[b] * edges[b+1])``.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import Optional

import numpy as np

SEED_BASE = 260307917
# Order in which child streams are spawned; never reorder (changes every input).
STREAMS = ("centres", "cluster_params", "assignment", "noise", "lengths",
           "queries", "prompt_lengths", "masses", "standing", "attained", "trace",
           "hist_prompt_lengths")


def streams(config_id: int, seed_base: int = SEED_BASE) -> dict:
    ss = np.random.SeedSequence([seed_base, int(config_id)])
    children = ss.spawn(len(STREAMS))
    return {name: np.random.default_rng(c) for name, c in zip(STREAMS, children)}


@dataclass
class PromptLenSpec:
    kind: str                 # "uniform" (lo..hi inclusive) or "lognormal"
    a: float                  # lo, or mu
    b: float                  # hi, or sigma
    lo: int = 1
    hi: int = 1 << 30


@dataclass
class PredictSpec:
    """A batch of pending requests scored against a history store."""
    Q: int
    N: int
    d: int
    clusters: int
    mu_range: tuple
    s_range: tuple
    L_max: int
    k: int
    B: int
    tau: float = 0.8
    prompt: PromptLenSpec = field(default_factory=lambda: PromptLenSpec("uniform", 16, 2048))
    sigma: float = 0.3
    sigma_per_coordinate: bool = False
    noise_frac: float = 0.0
    zipf: Optional[float] = None


@dataclass
class IndexSpec:
    """Requests that already carry a length distribution (cost/index/rank only)."""
    Q: int
    B: int
    L_max: int
    alpha: float
    prompt: PromptLenSpec
    tiny: float = 1e-30


CONFIGS = {
    1: PredictSpec(Q=256, N=8192, d=384, clusters=32, mu_range=(3.0, 6.0), s_range=(0.5, 1.0),
                   L_max=4096, k=32, B=128, prompt=PromptLenSpec("uniform", 16, 2048, 16, 2048)),
    2: PredictSpec(Q=4096, N=262144, d=768, clusters=256, mu_range=(3.0, 7.0), s_range=(0.4, 1.2),
                   L_max=8192, k=64, B=256, prompt=PromptLenSpec("lognormal", 6.0, 1.0, 8, 8192)),
    3: PredictSpec(Q=16384, N=1048576, d=1024, clusters=1024, mu_range=(3.0, 7.0), s_range=(0.4, 1.2),
                   L_max=16384, k=64, B=256, noise_frac=0.1,
                   prompt=PromptLenSpec("lognormal", 6.0, 1.0, 8, 16384)),
    4: IndexSpec(Q=65536, B=1024, L_max=32768, alpha=0.1,
                 prompt=PromptLenSpec("lognormal", 7.0, 1.2, 8, 32768)),
    # Streaming case: 1,024 calls of 8 new requests each against a standing
    # queue of 8,192; Q below is the total number of new requests.
    5: PredictSpec(Q=1024 * 8, N=4194304, d=768, clusters=4096, mu_range=(2.0, 8.0),
                   s_range=(0.3, 1.5), L_max=32768, k=128, B=512, zipf=1.1,
                   prompt=PromptLenSpec("lognormal", 6.0, 1.0, 8, 32768)),
}

WORKLOAD_NAMES = {
    1: "tiny: Q=256 N=8192 d=384 k=32 B=128",
    2: "mid: Q=4096 N=262144 d=768 k=64 B=256",
    3: "gemm-bound: Q=16384 N=1048576 d=1024 k=64 B=256 (10% noise rows)",
    4: "index-bound: Q=65536 B=1024 Dirichlet(0.1) masses",
    5: "streaming: 1024 calls x 8 queries, N=4194304 d=768 k=128 B=512",
}


def log_bins(L_max: int, B: int):
    """Bin edges ``L_max**(b/B)`` (b = 0..B) and geometric-centre representatives."""
    b = np.arange(B + 1, dtype=np.float64)
    edges = np.power(float(L_max), b / float(B))
    edges[0] = 1.0
    edges[-1] = float(L_max)
    repr_ = np.sqrt(edges[:-1] * edges[1:])
    return edges, repr_


def _prompt_lengths(rng, spec: PromptLenSpec, n: int) -> np.ndarray:
    if spec.kind == "uniform":
        x = rng.integers(int(spec.a), int(spec.b) + 1, size=n)
    elif spec.kind == "lognormal":
        x = np.rint(np.exp(rng.normal(spec.a, spec.b, size=n)))
    else:
        raise ValueError(spec.kind)
    return np.clip(x, spec.lo, spec.hi).astype(np.int32)


def _unit_rows(x: np.ndarray) -> np.ndarray:
    return x / np.linalg.norm(x, axis=1, keepdims=True)


@dataclass
class PredictInputs:
    spec: PredictSpec
    hist_emb: np.ndarray      # [N, d] float32, unit rows
    hist_len: np.ndarray      # [N] int32
    hist_cluster: np.ndarray  # [N] int32 (-1 for noise rows)
    queries: np.ndarray       # [Q, d] float32
    query_cluster: np.ndarray # [Q] int32
    prompt_len: np.ndarray    # [Q] int32
    bin_edges: np.ndarray     # [B+1] float64
    bin_repr: np.ndarray      # [B] float64
    seed: list
    hist_prompt_len: Optional[np.ndarray] = None   # [N] int32: input lengths of the stored records


def _cluster_probs(spec: PredictSpec, rng) -> np.ndarray:
    if spec.zipf is None:
        return np.full(spec.clusters, 1.0 / spec.clusters)
    ranks = np.arange(1, spec.clusters + 1, dtype=np.float64)
    p = ranks ** (-spec.zipf)
    p /= p.sum()
    return p[rng.permutation(spec.clusters)]   # popularity ranks shuffled over clusters


def _points(rng, centres, assign, spec: PredictSpec, noise_mask, block=65536) -> np.ndarray:
    """Unit rows around the assigned centres (noise rows: uniform on the sphere).

    Block i of `block` rows draws from its own child of rng's seed sequence, so
    the blocks are generated in parallel threads and the result does not depend
    on the thread count.
    """
    import os
    from concurrent.futures import ThreadPoolExecutor
    n, d = assign.shape[0], centres.shape[1]
    out = np.empty((n, d), dtype=np.float32)
    scale = np.float32(spec.sigma if spec.sigma_per_coordinate else spec.sigma / np.sqrt(d))
    c32 = centres.astype(np.float32)
    n_blocks = (n + block - 1) // block
    kids = rng.bit_generator.seed_seq.spawn(n_blocks)

    def work(i):
        s, e = i * block, min(n, (i + 1) * block)
        g = np.random.default_rng(kids[i]).standard_normal((e - s, d), dtype=np.float32)
        x = c32[np.maximum(assign[s:e], 0)]
        x += scale * g
        nm = noise_mask[s:e]
        x[nm] = g[nm]                       # uniform on the sphere after normalising
        x /= np.linalg.norm(x, axis=1, keepdims=True)
        out[s:e] = x

    threads = max(1, min(16, os.cpu_count() or 1, n_blocks))
    with ThreadPoolExecutor(threads) as ex:
        list(ex.map(work, range(n_blocks)))
    return out


def make_predict(spec: PredictSpec, config_id: int, seed_base: int = SEED_BASE) -> PredictInputs:
    r = streams(config_id, seed_base)
    centres = _unit_rows(r["centres"].standard_normal((spec.clusters, spec.d)))
    mus = r["cluster_params"].uniform(*spec.mu_range, size=spec.clusters)
    ss = r["cluster_params"].uniform(*spec.s_range, size=spec.clusters)
    probs = _cluster_probs(spec, r["cluster_params"])

    ra = r["assignment"]
    hist_cluster = ra.choice(spec.clusters, size=spec.N, p=probs).astype(np.int32)
    hist_noise = ra.random(spec.N) < spec.noise_frac
    law = np.where(hist_noise, ra.integers(0, spec.clusters, size=spec.N), hist_cluster)
    hist_cluster = np.where(hist_noise, -1, hist_cluster).astype(np.int32)
    hist_emb = _points(r["noise"], centres, hist_cluster, spec, hist_noise)

    z = r["lengths"].standard_normal(spec.N)
    hist_len = np.clip(np.rint(np.exp(mus[law] + ss[law] * z)), 1, spec.L_max).astype(np.int32)

    rq = r["queries"]
    q_cluster = rq.choice(spec.clusters, size=spec.Q, p=probs).astype(np.int32)
    q_noise = rq.random(spec.Q) < spec.noise_frac
    q_cluster = np.where(q_noise, -1, q_cluster).astype(np.int32)
    queries = _points(rq, centres, q_cluster, spec, q_noise)

    prompt_len = _prompt_lengths(r["prompt_lengths"], spec.prompt, spec.Q)
    # Input lengths of the stored records, from the same law as the pending
    # requests' and independent of everything else (the stand-in data carry
    # no relation between input and output length).
    hist_prompt_len = _prompt_lengths(r["hist_prompt_lengths"], spec.prompt, spec.N)
    edges, repr_ = log_bins(spec.L_max, spec.B)
    return PredictInputs(spec, hist_emb, hist_len, hist_cluster, queries, q_cluster,
                         prompt_len, edges, repr_, [seed_base, config_id], hist_prompt_len)


@dataclass
class IndexInputs:
    spec: IndexSpec
    mass: np.ndarray          # [Q, B] float32 (rows sum to ~1; not renormalised after the cast)
    prompt_len: np.ndarray    # [Q] int32
    bin_edges: np.ndarray
    bin_repr: np.ndarray
    seed: list


def make_index(spec: IndexSpec, config_id: int, seed_base: int = SEED_BASE,
               block: int = 8192) -> IndexInputs:
    r = streams(config_id, seed_base)
    mass = np.empty((spec.Q, spec.B), dtype=np.float32)
    for s in range(0, spec.Q, block):
        e = min(spec.Q, s + block)
        g = r["masses"].gamma(spec.alpha, size=(e - s, spec.B))
        p = g / g.sum(axis=1, keepdims=True)
        p[p < spec.tiny] = 0.0
        mass[s:e] = p.astype(np.float32)
    prompt_len = _prompt_lengths(r["prompt_lengths"], spec.prompt, spec.Q)
    edges, repr_ = log_bins(spec.L_max, spec.B)
    return IndexInputs(spec, mass, prompt_len, edges, repr_, [seed_base, config_id])


def make_standing(spec: PredictSpec, config_id: int, n: int, seed_base: int = SEED_BASE):
    """The streaming workload's standing queue: n more requests from the same
    mixture (embeddings and prompt lengths), drawn from the "standing" stream.
    Returns (queries [n, d] float32, prompt_len [n] int32)."""
    r = streams(config_id, seed_base)
    centres = _unit_rows(r["centres"].standard_normal((spec.clusters, spec.d)))
    cp = r["cluster_params"]
    cp.uniform(*spec.mu_range, size=spec.clusters)      # same draws as make_predict
    cp.uniform(*spec.s_range, size=spec.clusters)
    probs = _cluster_probs(spec, cp)
    rs = r["standing"]
    q_cluster = rs.choice(spec.clusters, size=n, p=probs).astype(np.int32)
    q_noise = rs.random(n) < spec.noise_frac
    q_cluster = np.where(q_noise, -1, q_cluster).astype(np.int32)
    queries = _points(rs, centres, q_cluster, spec, q_noise)
    prompt_len = _prompt_lengths(rs, spec.prompt, n)
    return queries, prompt_len


def generated_tokens(config_id: int, Q: int, L_max: int, running: float = 0.5,
                     seed_base: int = SEED_BASE) -> np.ndarray:
    """Output tokens already generated by each request (0 for those not yet
    started): a fraction `running` of the requests are running, with
    floor(L_max * u^2 / 4), u ~ U(0, 1), tokens so far. int32 [Q]."""
    r = streams(config_id, seed_base)["attained"]
    run = r.random(Q) < running
    u = r.random(Q)
    return np.where(run, np.floor(L_max * u * u / 4.0), 0).astype(np.int32)


@dataclass
class TraceInputs:
    """A stream of requests for the queueing simulation."""
    arrival: np.ndarray       # [R] float64 seconds, non-decreasing (Poisson process)
    queries: np.ndarray       # [R, d] float32 prompt embeddings
    cluster: np.ndarray       # [R] int32 (-1 for noise requests)
    prompt_len: np.ndarray    # [R] int32 input lengths I
    output_len: np.ndarray    # [R] int32 true output lengths O (unknown to the scheduler)
    rps: float


def make_trace(spec: PredictSpec, config_id: int, R: int, rps: float,
               seed_base: int = SEED_BASE) -> TraceInputs:
    """R requests of the mixture behind a history store, arriving as a Poisson
    process of rate ``rps`` (Sec. 4.1 draws submission intervals from a
    Poisson process). Each request belongs to a cluster drawn like the store's
    rows; its true output length follows that cluster's lognormal law, so the
    store's neighbours of its prompt carry its length distribution. Drawn
    from the "trace" stream; the cluster centres and laws are the store's."""
    r = streams(config_id, seed_base)
    centres = _unit_rows(r["centres"].standard_normal((spec.clusters, spec.d)))
    cp = r["cluster_params"]
    mus = cp.uniform(*spec.mu_range, size=spec.clusters)
    ss = cp.uniform(*spec.s_range, size=spec.clusters)
    probs = _cluster_probs(spec, cp)
    rt = r["trace"]
    arrival = np.cumsum(rt.exponential(1.0 / float(rps), size=R))
    cluster = rt.choice(spec.clusters, size=R, p=probs).astype(np.int32)
    noise = rt.random(R) < spec.noise_frac
    law = np.where(noise, rt.integers(0, spec.clusters, size=R), cluster)
    cluster = np.where(noise, -1, cluster).astype(np.int32)
    queries = _points(rt, centres, cluster, spec, noise)
    prompt_len = _prompt_lengths(rt, spec.prompt, R)
    z = rt.standard_normal(R)
    output_len = np.clip(np.rint(np.exp(mus[law] + ss[law] * z)), 1, spec.L_max).astype(np.int32)
    return TraceInputs(arrival, queries, cluster, prompt_len, output_len, float(rps))


def make_config(config_id: int, **overrides):
    """Inputs of one of the five named workloads; keyword overrides shrink it."""
    base = CONFIGS[config_id]
    spec = type(base)(**{**base.__dict__, **overrides})
    if isinstance(spec, IndexSpec):
        return make_index(spec, config_id)
    return make_predict(spec, config_id)


def small_predict(Q, N, d, k, B, *, seed, clusters=8, L_max=4096, tau=0.8,
                  noise_frac=0.0, zipf=None, mu_range=(3.0, 6.0), s_range=(0.5, 1.0),
                  sigma=0.3, prompt=None) -> PredictInputs:
    """A custom-sized mixture for tests (seeded by ``seed``, not a config id)."""
    spec = PredictSpec(Q=Q, N=N, d=d, clusters=clusters, mu_range=mu_range, s_range=s_range,
                       L_max=L_max, k=k, B=B, tau=tau, sigma=sigma, noise_frac=noise_frac,
                       zipf=zipf, prompt=prompt or PromptLenSpec("uniform", 16, 2048, 16, 2048))
    return make_predict(spec, 100000 + int(seed))


def small_index(Q, B, *, seed, L_max=32768, alpha=0.1) -> IndexInputs:
    spec = IndexSpec(Q=Q, B=B, L_max=L_max, alpha=alpha,
                     prompt=PromptLenSpec("lognormal", 7.0, 1.2, 8, L_max))
    return make_index(spec, 100000 + int(seed))
