"""The streaming workload end to end: a standing queue of 8,192 requests over
the 4M-row store; each decision admits 8 new requests, re-indexes all 8,200,
ranks them and dispatches 8. The new requests are checked against the
oracle's own predictions and indices on a few decisions; the queue mechanics
(slot refills, re-index, stable rank) by their properties."""
import numpy as np
import pytest
import torch

import oracle
from paper_2603_07917_amd import sage, workloads
from tests import parity

pytestmark = pytest.mark.gpu


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def host(t):
    torch.cuda.synchronize()
    return t.cpu().numpy()


def oracle_rows(queries_f32, hist_f32, block=1 << 18):
    """fp64 score rows of a few queries over the whole store, in row blocks."""
    qb = oracle.round_to_bf16(queries_f32)
    parts = [oracle.similarity(qb, oracle.round_to_bf16(hist_f32[s:s + block]))
             for s in range(0, hist_f32.shape[0], block)]
    return np.concatenate(parts, axis=1)


def test_streaming_decisions_vs_oracle():
    spec = workloads.CONFIGS[5]
    batch, standing = 8, 8192
    w = workloads.make_config(5)
    sq, splen = workloads.make_standing(spec, 5, standing)
    print("workload generated", flush=True)
    store = sage.Store(dev(w.hist_emb), dev(w.hist_len), dev(w.bin_edges), dev(w.bin_repr),
                       spec.k, spec.tau)
    _, _, _, smass = store.predict(dev(sq))
    queue = sage.Queue(store, smass.clone(), dev(splen), batch)
    requests = list(range(standing))                  # queued request ids in slot order
    for call in range(3):
        a = call * batch
        q_new = w.queries[a:a + batch]
        p_new = w.prompt_len[a:a + batch]
        free_before = host(queue.free).copy()
        (ids, sims, counts, mass), dispatched = queue.decide(dev(q_new), dev(p_new))
        ids, sims, counts, mass = host(ids), host(sims), host(counts), host(mass)
        # the new requests' predictions against the oracle's own
        S = oracle_rows(q_new, w.hist_emb)
        clean, mass_o, delta = parity.check_predict(ids, sims, counts, mass, S, w.hist_len,
                                                    w.bin_edges, spec.tau, spec.k)
        # they went into the freed slots
        qmass, qplen = host(queue.mass), host(queue.prompt_len)
        assert np.array_equal(qmass[free_before], mass)
        assert np.array_equal(qplen[free_before], p_new)
        g, order = host(queue.index), host(queue.order)
        # the new requests' index against the oracle's, from the oracle's masses
        parity.check_index_downstream(g[free_before], mass_o, oracle.cost(p_new, w.bin_repr), delta,
                                      np.nonzero(clean)[0])
        # every slot was re-indexed from the queue's current masses, then ranked stably
        g_again = host(sage.index(queue.mass, queue.prompt_len, store.bin_repr))
        assert np.array_equal(g.view(np.uint32), g_again.view(np.uint32))
        parity.check_sorted_stably(order, g)
        # dispatch: the first `batch` slots of the order, by request id
        for j, slot in enumerate(free_before):
            if slot >= len(requests):
                requests.append(None)
            requests[slot] = standing + a + j
        want = [requests[s] for s in order[:batch]]
        assert list(host(dispatched)) == want
        assert np.array_equal(host(queue.free), order[:batch])
        print(f"call {call}: {int(clean.sum())}/{batch} rows compared through the index; "
              f"dispatched {want}", flush=True)
