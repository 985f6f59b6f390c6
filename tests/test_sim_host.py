"""The native event loop (sage_simulate, host code in libsage) against the
oracle's simulation: the same trace and the same priority order must give
identical completion times and preemption counts. Both evaluate the same
fp64 expressions (segment start + remaining service / rate), so the
comparison is exact. The orders here are seeded random permutations (the
ranking that produces real orders is tested on the GPU)."""
from __future__ import annotations

import numpy as np
import pytest

import oracle
from oracle import sage_sim

sage = pytest.importorskip("paper_2603_07917_amd.sage")


@pytest.fixture(scope="module")
def lib():
    try:
        return sage.load_library()
    except sage.SageError as e:
        pytest.skip(str(e))


def _trace(R, rps, seed, O_hi=300, I_hi=400):
    rng = np.random.default_rng(seed)
    arrival = np.cumsum(rng.exponential(1.0 / rps, size=R))
    I = rng.integers(0, I_hi + 1, size=R).astype(np.int32)
    O = np.maximum(1, np.rint(np.exp(rng.normal(3.5, 1.0, size=R)))).clip(1, O_hi).astype(np.int32)
    return arrival, I, O, rng


CASES = [  # (R, servers, load, queue_cap, bucket)
    (1, 1, 0.5, 10, 0),
    (2000, 1, 0.9, 1000, 0),
    (2000, 1, 0.95, 5, 0),
    (2000, 4, 0.9, 1000, 0),
    (1500, 1, 0.9, 1000, 16),
    (1500, 3, 0.97, 0, 16),
    (1500, 2, 1.3, 20, 50),          # overloaded: the backlog outside grows
    (600, 8, 0.8, 3, 1),
]


@pytest.mark.parametrize("R,servers,load,cap,bucket", CASES)
def test_matches_oracle(lib, R, servers, load, cap, bucket):
    arrival, I, O, rng = _trace(R, 8.0 * servers, seed=R + 31 * servers + bucket)
    rate = 8.0 * servers * oracle.service_cost(I, O).mean() / (servers * load)
    levels = sage_sim.refresh_levels(O, bucket) if bucket else 1
    order = rng.permutation(levels * R).astype(np.int32)
    # with refreshing, the last fifth of the positions carry no information
    informed = levels * R - (levels * R) // 5 if bucket else R
    f0, p0 = oracle.simulate(arrival, I, O, order, servers=servers, rate=rate, queue_cap=cap,
                             bucket=bucket, levels=levels, informed=informed)
    f1, p1 = sage.simulate(arrival, I, O, order, servers=servers, rate=rate, queue_cap=cap,
                           bucket=bucket, levels=levels, informed=informed)
    assert np.array_equal(f1, f0)
    assert np.array_equal(p1, p0)


def test_fcfs_and_ties(lib):
    # simultaneous arrivals and an arrival at a completion instant
    arrival = np.array([0.0, 0.0, 0.0, 1.0, 1.0, 3.0])
    I = np.array([0, 2, 1, 0, 0, 4], np.int32)
    O = np.array([2, 1, 2, 1, 4, 1], np.int32)          # C = 2, 2.5, 4, 0.5, 8, 4.5
    for order in (np.arange(6), np.array([5, 3, 1, 0, 4, 2]), np.array([4, 2, 0, 1, 3, 5])):
        for servers in (1, 2):
            f0, p0 = oracle.simulate(arrival, I, O, order, servers=servers, rate=1.0, queue_cap=1)
            f1, p1 = sage.simulate(arrival, I, O, order.astype(np.int32), servers=servers, rate=1.0,
                                   queue_cap=1)
            assert np.array_equal(f1, f0) and np.array_equal(p1, p0)


def test_hand_refresh(lib):
    f, p = sage.simulate([0.0, 1.0], [0, 0], [4, 2], [1, 2, 3, 4, 0, 5, 6, 7], rate=1.0, servers=1,
                         queue_cap=10, bucket=1, levels=4)
    assert f.tolist() == [10.0, 4.0] and p.tolist() == [2, 1]


def test_hand_uninformed_refresh(lib):
    arr, I, O, order = [0.0, 1.0], [0, 0], [3, 1], [0, 1, 2, 3, 4, 5]
    f, p = sage.simulate(arr, I, O, order, rate=1.0, queue_cap=4, bucket=1, levels=3)
    assert f.tolist() == [5.0, 1.5] and p.tolist() == [1, 0]
    f, p = sage.simulate(arr, I, O, order, rate=1.0, queue_cap=4, bucket=1, levels=3, informed=2)
    assert f.tolist() == [4.5, 5.0] and p.tolist() == [0, 0]


def test_empty_trace(lib):
    f, p = sage.simulate(np.zeros(0), np.zeros(0), np.zeros(0), np.zeros(0), rate=1.0)
    assert f.shape == (0,) and p.shape == (0,)


@pytest.mark.parametrize("kw,msg", [
    (dict(order=[0, 0, 2]), "permutation"),
    (dict(order=[0, 1, 3]), "permutation"),
    (dict(arrival=[0.0, 2.0, 1.0]), "decrease"),
    (dict(arrival=[0.0, np.nan, 1.0]), "finite"),
    (dict(output_len=[1, 0, 2]), "output_len"),
    (dict(prompt_len=[1, -1, 2]), "prompt_len"),
    (dict(rate=0.0), "rate"),
    (dict(rate=np.inf), "rate"),
    (dict(servers=0), "servers"),
    (dict(queue_cap=-1), "queue_cap"),
    (dict(bucket=1), "levels"),                  # O = 2 needs two levels with bucket 1
    (dict(levels=2, order=list(range(6))), "bucket 0"),
    (dict(informed=4), "informed"),
    (dict(informed=-1), "informed"),
])
def test_validation(lib, kw, msg):
    args = dict(arrival=[0.0, 1.0, 1.0], prompt_len=[1, 1, 1], output_len=[1, 2, 1], order=[2, 0, 1],
                rate=1.0, servers=1, queue_cap=4, bucket=0, levels=1, informed=None)
    args.update(kw)
    with pytest.raises(sage.SageError, match=msg):
        sage.simulate(args.pop("arrival"), args.pop("prompt_len"), args.pop("output_len"),
                      args.pop("order"), **args)
