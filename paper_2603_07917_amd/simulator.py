"""TTLT of queue orderings on a request trace, computed through libsage.

The GPU does the data-parallel work once for the whole trace:

* the predicted length distribution of every request (``sage_predict``
  against a resident history store);
* per policy, one index value per request, or per (request, refresh level)
  for the refreshed Gittins order (``sage_index``, ``sage_index_variant``,
  ``sage_index_attained`` at k * bucket generated tokens, one launch per
  level), and one ``sage_rank`` over those values.

A refreshed index depends only on the request's own distribution, prompt
length and generated tokens, and a request only ever reaches the levels
below ceil(O / bucket); so the full table, ranked once, holds every
comparison the scheduler will make, and the replay compares integer keys.
The replay itself is ``sage_simulate`` (host event loop).

Policies (Sec. 4.3 baselines and ablations): ``fcfs`` (arrival order),
``mean`` (mean of the predicted cost distribution), ``gittins-static`` (the
index at arrival, never refreshed), ``gittins`` (refreshed at every bucket
boundary, Sec. 3.3).
"""
from __future__ import annotations

import math
import time
from dataclasses import dataclass, field

import numpy as np
import torch

from . import sage

POLICIES = ("fcfs", "mean", "gittins-static", "gittins")


def refresh_levels(output_len, bucket: int) -> int:
    """Levels of the refresh table: 0 .. ceil(max O / bucket) - 1."""
    if len(output_len) == 0:
        return 1
    return max(1, int(math.ceil(int(np.max(output_len)) / int(bucket))))


def rate_for_load(prompt_len, output_len, rps: float, servers: int, load: float) -> float:
    """Service rate (cost units per second per server) at which the trace's
    offered load is `load`: rps * mean(C) / (servers * rate) = load."""
    I = np.asarray(prompt_len, dtype=np.float64)
    O = np.asarray(output_len, dtype=np.float64)
    return float(rps) * float(np.mean(O * O / 2.0 + I * O)) / (int(servers) * float(load))


def policy_order(policy: str, mass: torch.Tensor, prompt_len: torch.Tensor, bin_repr: torch.Tensor,
                 arrival: np.ndarray, output_len: np.ndarray, bucket: int = 200, noise: float = 0.0):
    """Order of one policy on the device: returns (order int32 [levels * R], levels,
    informed), informed being the number of finite index values (the +inf
    entries of exhausted predictions rank last and carry no information).
    With noise = w > 0 the distributions are first merged with the uniform one
    at w : (1 - w) (the paper's inaccurate predictions, w = 0.2 for 1:4)."""
    R = mass.shape[0]
    dev = mass.device
    if policy == "fcfs":
        t = torch.from_numpy(np.asarray(arrival, dtype=np.float32)).to(dev)
        return sage.rank(t), 1, R
    if noise > 0.0:
        mass = sage.mix_uniform(mass, noise)
    if policy == "mean":
        return sage.rank(sage.index_variant(mass, prompt_len, bin_repr, kind="mean")), 1, R
    if policy == "gittins-static":
        return sage.rank(sage.index(mass, prompt_len, bin_repr)), 1, R
    if policy == "gittins":
        L = refresh_levels(output_len, bucket)
        table = torch.empty((L, R), dtype=torch.float32, device=dev)
        gen = torch.empty(R, dtype=torch.int32, device=dev)
        for k in range(L):
            gen.fill_(k * int(bucket))
            sage.index_attained(mass, prompt_len, bin_repr, gen, bucket=int(bucket), out=table[k])
        order = sage.rank(table.view(-1))
        informed = int(np.isfinite(table.cpu().numpy()).sum())
        return order, L, informed
    raise sage.SageError(f"unknown policy {policy!r}")


@dataclass
class PolicyResult:
    ttlt: np.ndarray            # [R] seconds
    preemptions: np.ndarray     # [R]
    levels: int
    gpu_ms: float               # index + rank kernels of this policy
    replay_ms: float            # host event loop

    @property
    def mean_ttlt(self) -> float:
        return float(self.ttlt.mean()) if self.ttlt.size else 0.0


@dataclass
class Comparison:
    results: dict = field(default_factory=dict)   # policy -> PolicyResult
    predict_ms: float = 0.0
    rate: float = 0.0
    mass: object = None                            # [R, B] predicted distributions (device)

    def mean_ttlt(self) -> dict:
        return {p: r.mean_ttlt for p, r in self.results.items()}


def compare(mass: torch.Tensor, prompt_len: torch.Tensor, bin_repr: torch.Tensor, arrival, output_len, *,
            rate: float, servers: int = 1, queue_cap: int = 1000, bucket: int = 200,
            policies=POLICIES, noise: float = 0.0) -> Comparison:
    """Replay the trace under each policy, given the predicted distributions
    `mass` [R, B] (device) and prompt lengths (device); arrival and the true
    output lengths are host arrays."""
    arrival = np.asarray(arrival, dtype=np.float64)
    O = np.asarray(output_len, dtype=np.int32)
    I_host = prompt_len.cpu().numpy()
    out = Comparison(rate=float(rate))
    for pol in policies:
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        order, L, informed = policy_order(pol, mass, prompt_len, bin_repr, arrival, O, bucket, noise)
        order = order.cpu().numpy()
        t1 = time.perf_counter()
        finish, pre = sage.simulate(arrival, I_host, O, order, rate=rate, servers=servers,
                                    queue_cap=queue_cap, bucket=int(bucket) if pol == "gittins" else 0,
                                    levels=L, informed=informed)
        t2 = time.perf_counter()
        out.results[pol] = PolicyResult(finish - arrival, pre, L, 1e3 * (t1 - t0), 1e3 * (t2 - t1))
    return out


def compare_trace(store: sage.Store, queries: torch.Tensor, prompt_len: torch.Tensor, arrival,
                  output_len, *, rate: float, servers: int = 1, queue_cap: int = 1000,
                  bucket: int = 200, chunk: int = 16384, policies=POLICIES,
                  noise: float = 0.0) -> Comparison:
    """Predict every request's distribution on the store, then `compare`."""
    R = queries.shape[0]
    B = store.bin_edges.shape[0] - 1
    dev = queries.device
    n = min(R, chunk)
    mass = torch.empty((R, B), dtype=torch.float32, device=dev)
    ids = torch.empty((n, store.k), dtype=torch.int32, device=dev)
    sims = torch.empty((n, store.k), dtype=torch.float32, device=dev)
    counts = torch.empty((n, B), dtype=torch.int32, device=dev)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for s in range(0, R, chunk):
        e = min(R, s + chunk)
        store.predict(queries[s:e], out=(ids[:e - s], sims[:e - s], counts[:e - s], mass[s:e]))
    torch.cuda.synchronize()
    predict_ms = 1e3 * (time.perf_counter() - t0)
    out = compare(mass, prompt_len, store.bin_repr, arrival, output_len, rate=rate, servers=servers,
                  queue_cap=queue_cap, bucket=bucket, policies=policies, noise=noise)
    out.predict_ms = predict_ms
    out.mass = mass
    return out
