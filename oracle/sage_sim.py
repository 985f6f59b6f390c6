"""CPU oracle of the queueing simulation (test infrastructure only).

Only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may use this module; the product path never does.

What is simulated. Requests arrive over time (Sec. 4.1: Poisson submission
intervals) and wait in the scheduler's queue; each of ``servers`` identical
servers runs one request at a time, preemptively (Sec. 3.3: preemption is
enabled, its overhead taken as negligible). The service a request needs is
the unified cost of Sec. 3.2 at its true lengths, C = O^2/2 + I*O; a server
delivers ``rate`` cost units per second, and after g generated tokens a
request has received a(g) = g^2/2 + I*g. Its time-to-last-token (TTLT, the
paper's metric, Sec. 2) is its finish time minus its arrival time.

Order. The queue is ordered by a priority key: the smaller key is served
first. A request's key is that of an entry of a table of ``levels * R``
entries; entry ``e = k * R + r`` is request r after it has crossed k bucket
boundaries (a boundary every ``bucket`` generated tokens, Sec. 3.3: the index
of a running request is refreshed only there). Without refreshing
(``bucket = 0``) every request keeps its level-0 entry. The keys are the
positions of the entries in ``order``, the queue order produced by ranking.
Entries at positions ``informed`` and beyond carry no information: a
refreshed index is +inf when the predicted distribution has no mass left
above the service already received (every predicted length has been
outlived), and +inf ranks last. Reaching such a level leaves the request's
key as it was (reading: the refresh has no remaining-cost distribution to
act on, so the last index stands; ranking such requests last instead starves
them behind every newcomer).

Readings where the paper is silent (each listed with the simulator's design):

* a decision is taken after every arrival, completion and bucket boundary;
  events at the same instant are applied first (completions, then
  boundaries, then arrivals) and one decision follows;
* at a decision the ``servers`` admitted requests with the smallest keys run;
  a running request that is not among them is preempted and keeps its
  attained service (preempt-resume, zero overhead);
* the scheduler holds at most ``queue_cap`` waiting requests besides those
  on the servers (Sec. 4.4: up to 1,000 buffered); later arrivals wait,
  in arrival order, outside it and are admitted as requests finish; their
  TTLT still counts from their arrival;
* service accrues linearly within a run segment: a segment starts when a
  request starts or resumes at (t0, a0) or crosses a boundary (then a0 is
  the boundary's a(g) exactly), and at time t its attained service is
  min(a0 + (t - t0) * rate, next mark), the next mark being the next
  boundary's service or C. It finishes at t0 + (C - a0) / rate and crosses
  the next boundary at t0 + (a(g_next) - a0) / rate.

Pins: tests/test_oracle_sim.py (hand-worked schedules, Lindley's recursion,
the multi-server FCFS recursion, Smith's shortest-first rule by brute force,
work conservation across policies, the Pollaczek-Khinchine and Cobham
formulas, invariance of the refresh machinery under level-blind keys).
"""
from __future__ import annotations

import math

import numpy as np

from .sage_oracle import (attained_service, cost, gittins, gittins_attained, mean_index, mix_uniform,
                          rank)


def service_cost(prompt_len, output_len) -> np.ndarray:
    """True service of each request: C = O^2/2 + I*O (Sec. 3.2) in fp64."""
    I = np.asarray(prompt_len, dtype=np.float64)
    O = np.asarray(output_len, dtype=np.float64)
    return O * O / 2.0 + I * O


def _served(I: int, g: int) -> float:
    """Service received after g generated tokens: g^2/2 + I*g."""
    return g * g / 2.0 + I * g


def simulate(arrival, prompt_len, output_len, order, *, servers: int, rate: float,
             queue_cap: int, bucket: int = 0, levels: int = 1, informed: int | None = None):
    """Event-by-event simulation; returns (finish [R] float64, preemptions [R] int32)."""
    arrival = [float(v) for v in np.asarray(arrival, dtype=np.float64)]
    I = [int(v) for v in np.asarray(prompt_len)]
    O = [int(v) for v in np.asarray(output_len)]
    R = len(arrival)
    order = np.asarray(order, dtype=np.int64)
    if order.shape != (levels * R,) or sorted(order.tolist()) != list(range(levels * R)):
        raise ValueError("simulate: order must be a permutation of levels * R entries")
    if any(arrival[i] > arrival[i + 1] for i in range(R - 1)):
        raise ValueError("simulate: arrivals must be non-decreasing")
    if bucket > 0 and any(math.ceil(O[r] / bucket) - 1 >= levels for r in range(R)):
        raise ValueError("simulate: too few levels for the longest request")
    key = [0] * (levels * R)
    for pos, e in enumerate(order.tolist()):
        key[e] = pos
    if informed is None:
        informed = levels * R
    C = [O[r] * O[r] / 2.0 + I[r] * O[r] for r in range(R)]

    level = [0] * R             # boundaries crossed
    cur = key[:R]               # current key: the level-0 entry until a refresh replaces it
    attained = [0.0] * R        # service at the last stop (0 before the first start)
    finish = [0.0] * R
    preempt = [0] * R
    running = {}                # r -> [t0, a0, mark, t_done, t_mark]
    waiting = set()
    arrived = admitted = done = 0
    pool = 0                    # admitted and unfinished

    def priority(r):
        return cur[r]

    def start(r, t):
        a0 = attained[r]
        g_next = (level[r] + 1) * bucket
        if bucket > 0 and g_next < O[r]:
            a_next = _served(I[r], g_next)
            t_mark = t + (a_next - a0) / rate
            mark = a_next
        else:
            t_mark = math.inf
            mark = C[r]
        running[r] = [t, a0, mark, t + (C[r] - a0) / rate, t_mark]

    while done < R:
        cands = [arrival[arrived]] if arrived < R else []
        for seg in running.values():
            cands.append(min(seg[3], seg[4]))
        t = min(cands)
        for r in sorted(running):                       # completions
            if running[r][3] == t:
                finish[r] = t
                del running[r]
                pool -= 1
                done += 1
        for r in sorted(running):                       # bucket boundaries
            seg = running[r]
            if seg[4] == t:
                level[r] += 1
                attained[r] = seg[2]
                if key[level[r] * R + r] < informed:
                    cur[r] = key[level[r] * R + r]
                start(r, t)
        while arrived < R and arrival[arrived] == t:     # arrivals
            arrived += 1
        while admitted < arrived and pool < queue_cap + servers:
            waiting.add(admitted)
            admitted += 1
            pool += 1
        chosen = sorted(list(running) + list(waiting), key=priority)[:servers]
        for r in sorted(running):
            if r not in chosen:
                t0, a0, mark = running[r][0], running[r][1], running[r][2]
                attained[r] = min(a0 + (t - t0) * rate, mark)
                preempt[r] += 1
                del running[r]
                waiting.add(r)
        for r in chosen:
            if r not in running:
                waiting.discard(r)
                start(r, t)
    return np.array(finish, dtype=np.float64), np.array(preempt, dtype=np.int32)


# -------------------------------------------------------------- policies
POLICIES = ("fcfs", "mean", "gittins-static", "gittins")


def refresh_levels(output_len, bucket: int) -> int:
    """Rows of the refresh table: levels 0 .. ceil(max O / bucket) - 1."""
    return max(1, int(math.ceil(int(np.max(output_len)) / bucket)))


def policy_order(policy: str, arrival, mass, prompt_len, bin_repr, output_len=None, bucket: int = 0,
                 noise: float = 0.0):
    """Queue order of a policy, as (order, levels, informed).

    * ``fcfs``: arrival order (vLLM's default, Sec. 2);
    * ``mean``: the mean of the predicted cost distribution (Sec. 4.3);
    * ``gittins-static``: the Gittins index at arrival, never refreshed (the
      paper's "Gittins-minus" ablation, Sec. 4.3);
    * ``gittins``: the Gittins index of the remaining cost, refreshed at every
      bucket boundary (Sec. 3.3); the table's level k holds the index after
      k * bucket generated tokens, and ``informed`` counts its finite values.

    The index values order the queue; the order is taken on their fp32
    values (the precision the scheduling kernels emit), ties to the lower
    entry id. With ``noise`` = w > 0 the predicted distributions are first
    merged with the uniform one at w : (1 - w) (Sec. 4.3's inaccurate
    predictions, w = 0.2 for 1:4).
    """
    R = len(prompt_len)
    if policy == "fcfs":
        return rank(np.asarray(arrival, dtype=np.float64)), 1, R
    if noise > 0.0:
        mass = mix_uniform(mass, noise)
    x = cost(prompt_len, bin_repr)
    if policy == "mean":
        return rank(mean_index(mass, x).astype(np.float32)), 1, R
    if policy == "gittins-static":
        return rank(gittins(mass, x)[0].astype(np.float32)), 1, R
    if policy == "gittins":
        L = refresh_levels(output_len, bucket)
        table = np.empty((L, R), dtype=np.float32)
        for k in range(L):
            a = attained_service(prompt_len, np.full(R, k * bucket), bucket)
            table[k] = gittins_attained(mass, x, a)[0].astype(np.float32)
        return rank(table.ravel()), L, int(np.isfinite(table).sum())
    raise ValueError(f"policy_order: unknown policy {policy!r}")


def simulate_policy(policy: str, arrival, mass, prompt_len, bin_repr, output_len, *, servers: int,
                    rate: float, queue_cap: int, bucket: int = 200, noise: float = 0.0):
    """Order the queue by `policy` and simulate; returns (ttlt, preemptions)."""
    order, levels, informed = policy_order(policy, arrival, mass, prompt_len, bin_repr, output_len,
                                           bucket, noise)
    b = bucket if policy == "gittins" else 0
    finish, pre = simulate(arrival, prompt_len, output_len, order, servers=servers, rate=rate,
                           queue_cap=queue_cap, bucket=b, levels=levels, informed=informed)
    return finish - np.asarray(arrival, dtype=np.float64), pre
