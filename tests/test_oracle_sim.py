"""Pins of the queueing-simulation oracle (oracle/sage_sim.py).

The simulator is checked against what queueing theory fixes independently of
it: hand-worked schedules, Lindley's recursion for a FCFS server, the
start-time recursion of a FCFS multi-server queue, Smith's shortest-first
rule found by brute force over every order, work conservation (a single
server's busy periods do not depend on the order), the Pollaczek-Khinchine
mean for M/G/1 FCFS and Cobham's means for M/G/1 preemptive priority.
"""
from __future__ import annotations

import heapq
import itertools

import numpy as np
import pytest

import oracle
from oracle import sage_sim


# ------------------------------------------------------------ hand-worked
def test_hand_fcfs_single_server():
    # A: C = 2^2/2 + 4*2 = 10 at t=0; B: C = 1/2 + 2 = 2.5 at t=2; rate 1.
    f, p = oracle.simulate([0.0, 2.0], [4, 2], [2, 1], [0, 1], servers=1, rate=1.0, queue_cap=10)
    assert f.tolist() == [10.0, 12.5] and p.tolist() == [0, 0]


def test_hand_static_preemption():
    # B outranks A: A runs 0-2 (2 units), B runs 2-4.5, A resumes and needs 8 more.
    f, p = oracle.simulate([0.0, 2.0], [4, 2], [2, 1], [1, 0], servers=1, rate=1.0, queue_cap=10)
    assert f.tolist() == [12.5, 4.5] and p.tolist() == [1, 0]


def test_hand_refresh_at_boundaries():
    # A: I=0, O=4 (C=8, boundaries at a=0.5, 2, 4.5); B: I=0, O=2 at t=1 (C=2, boundary 0.5).
    # Entries e = k*2 + r; order B0 < A1 < B1 < A2 < A0 < B2 < A3 < B3.
    # t=0.5 A reaches level 1; t=1 B0 outranks A1: A stops with 1.0; t=1.5 B reaches
    # level 1, A1 outranks B1: B stops with 0.5; t=2.5 A reaches level 2, B1 outranks
    # A2: A stops with 2; B finishes at 2.5 + 1.5 = 4; A finishes at 4 + 6 = 10.
    order = [1, 2, 3, 4, 0, 5, 6, 7]
    f, p = oracle.simulate([0.0, 1.0], [0, 0], [4, 2], order, servers=1, rate=1.0, queue_cap=10,
                           bucket=1, levels=4)
    assert f.tolist() == [10.0, 4.0] and p.tolist() == [2, 1]


def test_hand_uninformed_refresh_keeps_the_key():
    # A: I=0, O=3 (C=4.5, boundaries at a=0.5 and 2); B: I=0, O=1 at t=1 (C=0.5).
    # Entries e = k*2 + r, order A0 < B0 < A1 < B1 < A2 < B2.
    order = [0, 1, 2, 3, 4, 5]
    arr, I, O = [0.0, 1.0], [0, 0], [3, 1]
    # Every entry informed: A refreshes to A1 at t=0.5, B0 outranks it at t=1 (A stops
    # with 1.0); B runs 1-1.5; A resumes, reaches level 2 at 2.5 and finishes at 5.
    f, p = oracle.simulate(arr, I, O, order, servers=1, rate=1.0, queue_cap=4, bucket=1, levels=3)
    assert f.tolist() == [5.0, 1.5] and p.tolist() == [1, 0]
    # Only the first two positions informed: A's refreshes carry no information, so A
    # keeps A0, which outranks B0; A runs to 4.5, then B.
    f, p = oracle.simulate(arr, I, O, order, servers=1, rate=1.0, queue_cap=4, bucket=1, levels=3,
                           informed=2)
    assert f.tolist() == [4.5, 5.0] and p.tolist() == [0, 0]


def test_hand_two_servers():
    # rate 2; A (C=8) at 0, B (C=4) at 1, C (C=1.5) at 2; C outranks B outranks A.
    # A runs 0-2 (4 units) and is preempted by C; C runs 2-2.75, A resumes 2.75-4.75;
    # B runs 1-3 on the other server.
    f, p = oracle.simulate([0.0, 1.0, 2.0], [0, 1, 1], [4, 2, 1], [2, 1, 0], servers=2, rate=2.0,
                           queue_cap=10)
    assert f.tolist() == [4.75, 3.0, 2.75] and p.tolist() == [1, 0, 0]


def test_hand_queue_cap():
    # A (C=10) at 0, B (C=0.5) at 1, C (C=0.5) at 1.2; C outranks B outranks A.
    arr, I, O, order = [0.0, 1.0, 1.2], [4, 0, 0], [2, 1, 1], [2, 1, 0]
    # No room besides the server: B and C wait outside, then enter in arrival order.
    f, p = oracle.simulate(arr, I, O, order, servers=1, rate=1.0, queue_cap=0)
    assert f.tolist() == [10.0, 10.5, 11.0] and p.tolist() == [0, 0, 0]
    # One waiting place: B preempts A at 1 and finishes at 1.5; C, kept outside until
    # then, enters at 1.5 and outranks A; A resumes at 2 with 9 units left.
    f, p = oracle.simulate(arr, I, O, order, servers=1, rate=1.0, queue_cap=1)
    assert f.tolist() == [11.0, 1.5, 2.0] and p.tolist() == [1, 0, 0]


def test_rejects_bad_inputs():
    with pytest.raises(ValueError):
        oracle.simulate([0.0, 1.0], [1, 1], [1, 1], [0, 0], servers=1, rate=1.0, queue_cap=1)
    with pytest.raises(ValueError):
        oracle.simulate([1.0, 0.0], [1, 1], [1, 1], [0, 1], servers=1, rate=1.0, queue_cap=1)
    with pytest.raises(ValueError):   # O = 5 with bucket 2 needs levels 0, 1, 2
        oracle.simulate([0.0], [1], [5], [0, 1], servers=1, rate=1.0, queue_cap=1, bucket=2, levels=2)


# ------------------------------------------------------------ recursions
def _trace(R, rps, seed, O_hi=60, I_hi=200):
    rng = np.random.default_rng(seed)
    arrival = np.cumsum(rng.exponential(1.0 / rps, size=R))
    return arrival, rng.integers(0, I_hi + 1, size=R), rng.integers(1, O_hi + 1, size=R)


def test_fcfs_single_server_is_lindley():
    arrival, I, O = _trace(3000, 8.0, 1)
    C = oracle.service_cost(I, O)
    rate = 8.0 * C.mean() / 0.85
    f, p = oracle.simulate(arrival, I, O, np.arange(3000), servers=1, rate=rate, queue_cap=10 ** 6)
    want = np.empty(3000)
    prev = 0.0
    for r in range(3000):
        prev = max(arrival[r], prev) + C[r] / rate
        want[r] = prev
    assert np.array_equal(f, want) and not p.any()


@pytest.mark.parametrize("cap", [0, 7, 10 ** 6])
def test_fcfs_multi_server_recursion(cap):
    arrival, I, O = _trace(2000, 24.0, 2)
    C = oracle.service_cost(I, O)
    c = 3
    rate = 24.0 * C.mean() / (0.9 * c)
    f, p = oracle.simulate(arrival, I, O, np.arange(2000), servers=c, rate=rate, queue_cap=cap)
    free = [0.0] * c
    want = np.empty(2000)
    for r in range(2000):
        s = max(arrival[r], heapq.heappop(free))
        want[r] = s + C[r] / rate
        heapq.heappush(free, want[r])
    assert np.array_equal(f, want) and not p.any()


def test_smith_rule_by_brute_force():
    # All requests present at t=0 on one server: the mean completion time is
    # smallest when the shortest go first (Smith 1956), and then equals
    # (1/R) sum_i sum_{j<=i} C_(j) / rate.
    I = np.array([3, 0, 7, 2, 5, 2])
    O = np.array([2, 5, 1, 3, 2, 4])
    C = oracle.service_cost(I, O)
    assert len(set(C.tolist())) == 6
    rate = 1.5
    means = {}
    for perm in itertools.permutations(range(6)):
        f, _ = oracle.simulate(np.zeros(6), I, O, np.array(perm), servers=1, rate=rate, queue_cap=6)
        means[perm] = f.mean()
    best = min(means, key=means.get)
    assert list(best) == np.argsort(C).tolist()
    assert means[best] == pytest.approx(np.cumsum(np.sort(C) / rate).mean(), rel=1e-14)


# ------------------------------------------------------------ invariants
def _busy_ends(arrival, finish):
    ends = []
    fs = np.sort(finish)
    for i, t in enumerate(fs):
        if np.searchsorted(arrival, t, side="right") == i + 1:
            ends.append(t)
    return np.array(ends)


@pytest.mark.parametrize("cap", [3, 10 ** 6])
def test_work_conservation(cap):
    arrival, I, O = _trace(1500, 8.0, 3)
    C = oracle.service_cost(I, O)
    rate = 8.0 * C.mean() / 0.8
    rng = np.random.default_rng(4)
    runs = [oracle.simulate(arrival, I, O, np.arange(1500), servers=1, rate=rate, queue_cap=cap)[0],
            oracle.simulate(arrival, I, O, rng.permutation(1500), servers=1, rate=rate, queue_cap=cap)[0]]
    L = sage_sim.refresh_levels(O, 16)
    f, p = oracle.simulate(arrival, I, O, rng.permutation(L * 1500), servers=1, rate=rate,
                           queue_cap=cap, bucket=16, levels=L)
    assert p.sum() > 100           # the random refresh keys do preempt
    runs.append(f)
    ref = _busy_ends(arrival, runs[0])
    assert len(ref) > 20
    for f in runs[1:]:
        e = _busy_ends(arrival, f)
        assert len(e) == len(ref)
        np.testing.assert_allclose(e, ref, rtol=1e-11)
    # work-conserving single server: the last completion is the same too
    assert all(abs(f.max() - runs[0].max()) <= 1e-11 * runs[0].max() for f in runs)


def test_refresh_with_level_blind_keys_is_static():
    arrival, I, O = _trace(800, 8.0, 5)
    C = oracle.service_cost(I, O)
    rate = 8.0 * C.mean() / 0.9
    rng = np.random.default_rng(6)
    static = rng.permutation(800)
    pos = np.empty(800, np.int64)
    pos[static] = np.arange(800)
    L = sage_sim.refresh_levels(O, 8)
    e = np.arange(L * 800)
    order = e[np.lexsort((e // 800, pos[e % 800]))]     # by request rank, then level
    f0, p0 = oracle.simulate(arrival, I, O, static, servers=2, rate=rate, queue_cap=50)
    f1, p1 = oracle.simulate(arrival, I, O, order, servers=2, rate=rate, queue_cap=50,
                             bucket=8, levels=L)
    assert p0.sum() > 20 and np.array_equal(p0, p1)
    np.testing.assert_allclose(f1, f0, rtol=1e-12)


# ------------------------------------------------------------ closed forms
def test_pollaczek_khinchine_fcfs():
    # M/G/1 FCFS: E[T] = E[S] + lam E[S^2] / (2 (1 - rho)).
    rng = np.random.default_rng(7)
    R, lam = 60000, 8.0
    arrival = np.cumsum(rng.exponential(1.0 / lam, size=R))
    I = rng.integers(0, 51, size=R)
    O = rng.integers(1, 41, size=R)
    grid_I, grid_O = np.meshgrid(np.arange(0, 51), np.arange(1, 41))
    Cg = oracle.service_cost(grid_I.ravel(), grid_O.ravel())
    rho = 0.6
    rate = lam * Cg.mean() / rho
    ES, ES2 = Cg.mean() / rate, (Cg ** 2).mean() / rate ** 2
    f, _ = oracle.simulate(arrival, I, O, np.arange(R), servers=1, rate=rate, queue_cap=R)
    want = ES + lam * ES2 / (2.0 * (1.0 - rho))
    assert (f - arrival).mean() == pytest.approx(want, rel=0.04)


def test_cobham_preemptive_priority():
    # M/G/1 preemptive-resume priority, class 1 over class 2 (FCFS within a class):
    # E[T_k] = E[S_k] / (1 - s_{k-1}) + sum_{i<=k} lam_i E[S_i^2] / (2 (1 - s_{k-1}) (1 - s_k)).
    rng = np.random.default_rng(8)
    R, lam1, lam2 = 80000, 0.4, 0.1
    arrival = np.cumsum(rng.exponential(1.0 / (lam1 + lam2), size=R))
    cls = (rng.random(R) >= lam1 / (lam1 + lam2)).astype(int)      # 0: class 1, 1: class 2
    I = np.where(cls == 0, 0, 1)
    O = np.where(cls == 0, 1, 2)                                   # C = 0.5 and 4
    ids = np.arange(R)
    order = np.concatenate([ids[cls == 0], ids[cls == 1]])
    f, p = oracle.simulate(arrival, I, O, order, servers=1, rate=1.0, queue_cap=R)
    T = f - arrival
    S1, S2 = 0.5, 4.0
    s1, s2 = lam1 * S1, lam1 * S1 + lam2 * S2
    T1 = S1 + lam1 * S1 ** 2 / (2 * (1 - s1))
    T2 = S2 / (1 - s1) + (lam1 * S1 ** 2 + lam2 * S2 ** 2) / (2 * (1 - s1) * (1 - s2))
    assert p[cls == 0].sum() == 0 and p[cls == 1].sum() > 1000
    assert T[cls == 0].mean() == pytest.approx(T1, rel=0.02)
    assert T[cls == 1].mean() == pytest.approx(T2, rel=0.05)


# ------------------------------------------------------------ policies
def _binned_law_trace(R, seed, B=64, L_max=2048):
    """Requests whose predicted distribution is exactly the law their true
    output length is drawn from (a lognormal binned on the log bins)."""
    rng = np.random.default_rng(seed)
    b = np.arange(B + 1, dtype=np.float64)
    edges = np.power(float(L_max), b / B)
    repr_ = np.sqrt(edges[:-1] * edges[1:])
    mu = rng.uniform(2.0, 6.5, size=R)
    s = rng.uniform(0.3, 1.5, size=R)
    from scipy.stats import norm
    cdf = norm.cdf((np.log(edges)[None, :] - mu[:, None]) / s[:, None])
    mass = np.diff(cdf, axis=1)
    mass /= mass.sum(axis=1, keepdims=True)
    # true length: a bin drawn from the law, its representative length
    u = rng.random(R)
    bins = (mass.cumsum(axis=1) < u[:, None]).sum(axis=1).clip(0, B - 1)
    O = np.maximum(1, np.rint(repr_[bins])).astype(np.int64)
    I = rng.integers(16, 512, size=R)
    return mass, I, O, repr_


def test_policy_orders():
    mass, I, O, repr_ = _binned_law_trace(300, 9)
    arrival = np.sort(np.random.default_rng(10).random(300)) * 40
    o_f, L, n = sage_sim.policy_order("fcfs", arrival, mass, I, repr_)
    assert L == 1 and n == 300 and np.array_equal(o_f, np.arange(300))
    x = oracle.cost(I, repr_)
    o_m, _, _ = sage_sim.policy_order("mean", arrival, mass, I, repr_)
    assert np.array_equal(o_m, np.argsort((mass * x).sum(1).astype(np.float32), kind="stable"))
    o_s, _, _ = sage_sim.policy_order("gittins-static", arrival, mass, I, repr_)
    o_g, L, n = sage_sim.policy_order("gittins", arrival, mass, I, repr_, O, bucket=64)
    assert L == sage_sim.refresh_levels(O, 64) > 1
    # the uninformed entries are the table's +inf values (no mass above the attained
    # service): those past the largest representative length, and they rank last
    assert 300 < n < L * 300
    # level 0 of the refresh table is the index at arrival
    lvl0 = o_g[o_g < 300]
    assert np.array_equal(lvl0, o_s)


def test_gittins_beats_fcfs_and_mean_with_true_laws():
    # With the true length laws as predictions, the refreshed Gittins order is
    # the optimal non-anticipating policy of an M/G/1 queue (Gittins 1989);
    # on one trace it must beat arrival order by far and the mean order too.
    R = 1500
    mass, I, O, repr_ = _binned_law_trace(R, 11)
    rng = np.random.default_rng(12)
    arrival = np.cumsum(rng.exponential(1.0 / 8.0, size=R))
    rate = 8.0 * oracle.service_cost(I, O).mean() / 0.9
    mean_ttlt = {}
    for pol in oracle.POLICIES:
        T, _ = oracle.simulate_policy(pol, arrival, mass, I, repr_, O, servers=1, rate=rate,
                                      queue_cap=1000, bucket=64)
        mean_ttlt[pol] = T.mean()
    assert mean_ttlt["gittins"] < 0.5 * mean_ttlt["fcfs"]
    assert mean_ttlt["gittins"] < mean_ttlt["mean"]
    assert mean_ttlt["gittins"] <= mean_ttlt["gittins-static"] * 1.02
