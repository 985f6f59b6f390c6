"""TTLT of queue orderings through libsage against the oracle's simulation.

Both sides start from the same seeded history store and request trace. The
GPU predicts every request's distribution, computes each policy's index
values (and the refreshed Gittins table) and ranks them; the host replays
the trace (sage_simulate). The oracle does all of it on its own in fp64.

Checks, in order:
* predict and index of every request against the oracle's (clean rows);
* each policy's order is a stable sort of its own GPU index values;
* the replay of the ORACLE's order by sage_simulate equals the oracle's own
  replay bit for bit (the event loop, on real orders);
* the mean TTLT of each policy agrees with the oracle's within 2%, and at
  least 95% of the requests have bit-identical TTLTs (where an index pair
  falls within the fp32 rounding the two orders may differ and change later
  decisions); policies the oracle separates come out in the same order.
"""
import numpy as np
import pytest
import torch

import oracle
from oracle import sage_sim
from paper_2603_07917_amd import sage, simulator, workloads
from tests import parity

pytestmark = pytest.mark.gpu


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def host(t):
    torch.cuda.synchronize()
    return t.cpu().numpy()


CASES = [  # (R, servers, load, queue_cap, bucket, noise)
    (1200, 1, 0.9, 1000, 200, 0.0),
    (1600, 4, 0.95, 40, 100, 0.0),
    (1200, 1, 0.9, 1000, 200, 0.2),       # the paper's 1:4 inaccurate predictions
]


@pytest.mark.parametrize("R,servers,load,cap,bucket,noise", CASES)
def test_ttlt_policies_vs_oracle(R, servers, load, cap, bucket, noise):
    print(f"case R={R} servers={servers} load={load} cap={cap} bucket={bucket} noise={noise}", flush=True)
    spec = workloads.PredictSpec(Q=1, N=6000, d=128, clusters=12, mu_range=(3.0, 6.5),
                                 s_range=(0.3, 1.0), L_max=4096, k=32, B=64)
    cid = 500000 + R
    w = workloads.make_predict(spec, cid)
    rps = 8.0 * servers
    tr = workloads.make_trace(spec, cid, R, rps)
    rate = rps * oracle.service_cost(tr.prompt_len, tr.output_len).mean() / (servers * load)

    # the GPU: predict, per-policy orders, host replay
    store = sage.Store(dev(w.hist_emb), dev(w.hist_len), dev(w.bin_edges), dev(w.bin_repr),
                       spec.k, spec.tau)
    ids, sims, counts, mass = [host(t) for t in store.predict(dev(tr.queries))]
    cmp = simulator.compare_trace(store, dev(tr.queries), dev(tr.prompt_len), tr.arrival,
                                  tr.output_len, rate=rate, servers=servers, queue_cap=cap,
                                  bucket=bucket, noise=noise)
    assert np.array_equal(host(cmp.mass), mass)

    # the oracle: its own prediction from the same inputs
    S = oracle.similarity(oracle.round_to_bf16(tr.queries), oracle.round_to_bf16(w.hist_emb))
    clean, mass_o, delta = parity.check_predict(ids, sims, counts, mass, S, w.hist_len, w.bin_edges,
                                                spec.tau, spec.k)
    rows = np.nonzero(clean)[0]
    x = oracle.cost(tr.prompt_len, w.bin_repr)
    g = host(sage.index(dev(mass), dev(tr.prompt_len), dev(w.bin_repr)))
    parity.check_index_downstream(g, mass_o, x, delta, rows)

    means_o = {}
    for pol in oracle.POLICIES:
        res = cmp.results[pol]
        # GPU order of this policy: a stable sort of its own index values
        order_g, L, n_g = simulator.policy_order(pol, dev(mass), dev(tr.prompt_len), dev(w.bin_repr),
                                                 tr.arrival, tr.output_len, bucket, noise)
        m_pol = dev(mass) if noise == 0.0 or pol == "fcfs" else sage.mix_uniform(dev(mass), noise)
        order_g = host(order_g)
        assert L == res.levels
        if pol == "fcfs":
            assert np.array_equal(order_g, np.arange(R))
        else:
            if pol == "mean":
                vals = sage.index_variant(m_pol, dev(tr.prompt_len), dev(w.bin_repr), kind="mean")
            elif pol == "gittins-static":
                vals = sage.index(m_pol, dev(tr.prompt_len), dev(w.bin_repr))
            else:
                vals = torch.stack([sage.index_attained(m_pol, dev(tr.prompt_len), dev(w.bin_repr),
                                                        dev(np.full(R, k * bucket, np.int32)), bucket)
                                    for k in range(L)]).view(-1)
            vals = host(vals)
            parity.check_sorted_stably(order_g, vals)
            assert n_g == int(np.isfinite(vals).sum())
        # the oracle's order and replay
        order_o, L_o, n_o = sage_sim.policy_order(pol, tr.arrival, mass_o, tr.prompt_len, w.bin_repr,
                                                  tr.output_len, bucket, noise)
        assert L_o == L
        b = bucket if pol == "gittins" else 0
        f_o, p_o = oracle.simulate(tr.arrival, tr.prompt_len, tr.output_len, order_o, servers=servers,
                                   rate=rate, queue_cap=cap, bucket=b, levels=L, informed=n_o)
        # the native event loop on the oracle's order: bit-exact
        f_n, p_n = sage.simulate(tr.arrival, tr.prompt_len, tr.output_len, order_o, rate=rate,
                                 servers=servers, queue_cap=cap, bucket=b, levels=L, informed=n_o)
        assert np.array_equal(f_n, f_o) and np.array_equal(p_n, p_o)
        T_o = f_o - tr.arrival
        means_o[pol] = T_o.mean()
        same = np.mean(res.ttlt == T_o)
        assert res.mean_ttlt == pytest.approx(means_o[pol], rel=0.02), pol
        assert same >= 0.95, (pol, same)
        print(f"{pol}: mean TTLT gpu {res.mean_ttlt:.4f} s, oracle {means_o[pol]:.4f} s, "
              f"{100 * same:.1f}% identical, {int(res.preemptions.sum())} preemptions", flush=True)
    # policies the oracle separates by more than 4% come out in the same order
    means_g = cmp.mean_ttlt()
    for a in means_o:
        for b in means_o:
            if means_o[a] < 0.96 * means_o[b]:
                assert means_g[a] < means_g[b], (a, b)
    assert means_o["gittins"] < means_o["fcfs"]
