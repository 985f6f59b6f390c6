"""The threshold pre-pass of the neighbour search (Sec. 3.1) and the exact
fallback behind it, plus the device check of the bin preconditions.

The pre-pass bounds each query's k-th best score from below by theta0, the
k-th largest maximum of sampled 16-row groups; the search keeps only scores
>= theta0. That is exact when each sampled maximum is a score the search
itself computes for that row, bit for bit. The hardest case puts the k best
rows in distinct groups of sampled steps, so that theta0 equals the k-th best
score exactly: a search whose fp32 scores came out one ulp lower than the
pre-pass's would drop them. A second set of tests raises theta0 from the host
(sage_debug_theta_floor) so that queries are left with fewer than min(k, N)
candidates; they must be answered by the exact path with unchanged results.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2603_07917_amd import sage, workloads
from tests import parity

pytestmark = pytest.mark.gpu

STREAM_MAX_D = 2048          # the stream path takes d up to this


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def host(t):
    torch.cuda.synchronize()
    return t.cpu().numpy()


def run_predict(w, k, tau=0.8):
    qb = sage.ingest_bf16(dev(w.queries), "panels")
    hb = sage.ingest_bf16(dev(w.hist_emb), "panels")
    ids, sims, counts, mass = sage.predict(qb, hb, dev(w.hist_len), k, tau, dev(w.bin_edges))
    return host(ids), host(sims), host(counts), host(mass)


def oracle_scores(w):
    return oracle.similarity(oracle.round_to_bf16(w.queries), oracle.round_to_bf16(w.hist_emb))


def sample_every(Q, N, d, k):
    """The pre-pass's step stride as the library plans it: every SR-th whole
    256-row step, SR chosen for >= 4k group maxima (16 per step), at most 128
    on the stream path (at most 16 queries), else at most 16 for k <= 64 on a
    store below 2^29 elements and 32 otherwise, and at most 512 sampled steps."""
    steps = N // 256
    L = max(64, 1 << (k - 1).bit_length())
    assert steps * 16 >= 8 * k, "store too small for a pre-pass"
    wide = Q > 16 and N * d >= (1 << 29)
    few = Q <= 16 and d <= STREAM_MAX_D and k <= 256
    sr_max = 128 if few else (16 if (L == 64 and not wide) else 32)
    sr = max(1, min(sr_max, steps * 16 // (4 * k)))
    while -(-steps // sr) > 512:
        sr += 1
    return sr


def plant_kth_equals_theta(w, q, k, sr):
    """Copies of query q's own embedding as history rows, one in each of the
    16 groups of sampled steps 0, SR, 2 SR, ... until there are k of them;
    copy j sits at row (j (5 + 2 q) + 5 q) % 16 of its group, so queries
    0, 1 and 2 never share a row. They are query q's k best rows (cosine 1
    against about 0.92 within a cluster), each the maximum of its sampled
    group, so theta0 is the k-th best score itself."""
    rows = []
    for j in range(k):
        s, g = divmod(j, 16)
        rows.append(s * sr * 256 + 16 * g + (j * (5 + 2 * q) + 5 * q) % 16)
    rows = np.array(rows)
    w.hist_emb[rows] = w.queries[q]
    return rows


@pytest.mark.parametrize("Q,k", [(1, 64), (8, 128), (16, 256), (5, 32), (64, 64), (300, 16)])
def test_theta_equals_kth_score(Q, k):
    """Q <= 16: the stream path; larger Q with k <= 64: the filtered path."""
    N, d = 262144, 128
    print(f"case Q={Q} k={k}", flush=True)
    w = workloads.small_predict(Q=Q, N=N, d=d, k=k, B=64, seed=500 + Q + k, clusters=8)
    sr = sample_every(Q, N, d, k)
    planted = {}
    for q in range(min(Q, 3)):                       # up to three queries, distinct rows each
        planted[q] = plant_kth_equals_theta(w, q, k, sr)
    for q in planted:
        assert len(set(planted[q].tolist())) == k
    ids, sims, counts, mass = run_predict(w, k)
    S = oracle_scores(w)
    parity.check_predict(ids, sims, counts, mass, S, w.hist_len, w.bin_edges, 0.8, k)
    for q, rows in planted.items():
        assert np.all(w.hist_emb[rows] == w.queries[q])
        assert set(ids[q].tolist()) == set(rows.tolist()), f"query {q}: its {k} copies are its neighbours"


@pytest.mark.parametrize("Q,k,layout", [(8, 64, "panels"), (8, 128, "panels"), (3, 256, "rows"),
                                        (300, 32, "panels"), (64, 64, "rows")])
def test_raised_theta_goes_to_exact_fallback(Q, k, layout):
    """theta0 raised from the host: queries with fewer than min(k, N)
    candidates take the exact path; results equal the oracle's and, where the
    fallback computes the same fp32 scores as the fast path (the filtered
    path), the unforced run's bit for bit."""
    N, d = 100000, 96
    print(f"case Q={Q} k={k} layout={layout}", flush=True)
    w = workloads.small_predict(Q=Q, N=N, d=d, k=k, B=64, seed=700 + Q + k, clusters=6)
    qb = sage.ingest_bf16(dev(w.queries), layout)
    hb = sage.ingest_bf16(dev(w.hist_emb), layout)
    hl, be = dev(w.hist_len), dev(w.bin_edges)
    base = [host(t) for t in sage.predict(qb, hb, hl, k, 0.8, be)]
    S = oracle_scores(w)
    kth = base[1][:, k - 1]
    floors = [float(np.median(kth)), 2.0]          # about half the queries, then all of them
    try:
        for floor in floors:
            sage.debug_theta_floor(floor)
            out = [host(t) for t in sage.predict(qb, hb, hl, k, 0.8, be)]
            sage.debug_theta_floor(-np.inf)
            parity.check_predict(*out, S, w.hist_len, w.bin_edges, 0.8, k)
            if Q > 16:
                for a, b in zip(base, out):
                    assert np.array_equal(a.view(np.uint8), b.view(np.uint8)), f"floor {floor}"
    finally:
        sage.debug_theta_floor(-np.inf)


def test_check_inputs_flags_each_precondition():
    edges, repr_ = workloads.log_bins(8192, 64)
    plen = np.array([0, 5, 8192, 17], dtype=np.int32)
    ok = sage.check_inputs(dev(edges), dev(repr_), dev(plen), sync=False)
    assert int(host(ok)[0]) == 0
    cases = []
    e = edges.copy(); e[10], e[11] = e[11], e[10]; cases.append((e, repr_, plen, 1))      # swapped edges
    e = edges.copy(); e[5] = e[4]; cases.append((e, repr_, plen, 1))                       # equal edges
    e = edges.copy(); e[-1] = np.nan; cases.append((e, repr_, plen, 1))                    # NaN edge
    r = repr_.copy(); r[30] = r[29] - 1.0; cases.append((edges, r, plen, 2))              # decreasing repr
    r = repr_.copy(); r[0] = -1.0; cases.append((edges, r, plen, 2))                      # negative repr
    r = repr_.copy(); r[-1] = np.inf; cases.append((edges, r, plen, 2))                   # infinite repr
    p = plen.copy(); p[2] = -3; cases.append((edges, repr_, p, 4))                         # negative I
    e = edges.copy(); e[1] = 0.0; r = repr_.copy(); r[3] = 0.0; p = plen.copy(); p[0] = -1
    cases.append((e, r, p, 7))                                                              # all three
    for e, r, p, bits in cases:
        st = sage.check_inputs(dev(e), dev(r), dev(p), sync=False)
        assert int(host(st)[0]) == bits
        with pytest.raises(sage.SageError):
            sage.check_inputs(dev(e), dev(r), dev(p))
    # one array at a time; B from whichever is given
    assert int(host(sage.check_inputs(None, dev(repr_), None, sync=False))[0]) == 0
    assert int(host(sage.check_inputs(dev(cases[0][0]), None, None, sync=False))[0]) == 1


def test_store_rejects_unsorted_bins():
    w = workloads.small_predict(Q=4, N=2000, d=64, k=8, B=32, seed=3, clusters=3)
    e = w.bin_edges.copy()
    e[7], e[8] = e[8], e[7]
    with pytest.raises(sage.SageError, match="bin edges"):
        sage.Store(dev(w.hist_emb), dev(w.hist_len), dev(e), dev(w.bin_repr), 8)
    r = w.bin_repr[::-1].copy()
    with pytest.raises(sage.SageError, match="representatives"):
        sage.Store(dev(w.hist_emb), dev(w.hist_len), dev(w.bin_edges), dev(r), 8)
    sage.Store(dev(w.hist_emb), dev(w.hist_len), dev(w.bin_edges), dev(w.bin_repr), 8)   # fine


@pytest.mark.parametrize("Q,k", [(300, 32), (8, 64)])
def test_fallback_word_from_an_earlier_call(Q, k):
    """One workspace for a call that flags queries (theta0 raised from the
    host) and then for calls that flag none: the later calls clear the word
    the flagging call set before their select runs, so their fallback
    launches return at once, and their results equal the oracle's and the
    first unforced call's bit for bit."""
    N, d = 60000, 64
    print(f"case Q={Q} k={k}", flush=True)
    w = workloads.small_predict(Q=Q, N=N, d=d, k=k, B=32, seed=900 + Q + k, clusters=5)
    qb = sage.ingest_bf16(dev(w.queries), "panels")
    hb = sage.ingest_bf16(dev(w.hist_emb), "panels")
    hl, be = dev(w.hist_len), dev(w.bin_edges)
    ws = torch.empty(sage.predict_workspace_bytes(Q, N, d, k, 32), dtype=torch.uint8, device="cuda")
    S = oracle_scores(w)
    base = [host(t) for t in sage.predict(qb, hb, hl, k, 0.8, be, workspace=ws)]
    parity.check_predict(*base, S, w.hist_len, w.bin_edges, 0.8, k)
    try:
        sage.debug_theta_floor(2.0)                  # every query flagged
        forced = [host(t) for t in sage.predict(qb, hb, hl, k, 0.8, be, workspace=ws)]
    finally:
        sage.debug_theta_floor(-np.inf)
    parity.check_predict(*forced, S, w.hist_len, w.bin_edges, 0.8, k)
    for _ in range(2):
        again = [host(t) for t in sage.predict(qb, hb, hl, k, 0.8, be, workspace=ws)]
        for a, b in zip(base, again):
            assert np.array_equal(a.view(np.uint8), b.view(np.uint8))


def test_timer_only_times_the_named_launches():
    w = workloads.small_predict(Q=64, N=20000, d=64, k=16, B=32, seed=11, clusters=4)
    qb = sage.ingest_bf16(dev(w.queries), "panels")
    hb = sage.ingest_bf16(dev(w.hist_emb), "panels")
    hl, be = dev(w.hist_len), dev(w.bin_edges)
    torch.cuda.synchronize()
    full = sage.StageTimer(capacity=256)
    with full:
        sage.predict(qb, hb, hl, 16, 0.8, be)
        torch.cuda.synchronize()
    names = set(full.totals())
    full.close()
    assert {"sim_topk", "hist"} <= names
    only = sage.StageTimer(capacity=256, only="hist")
    with only:
        sage.predict(qb, hb, hl, 16, 0.8, be)
        torch.cuda.synchronize()
    got = only.totals()
    only.close()
    assert set(got) == {"hist"} and got["hist"][0] == 1 and got["hist"][1] > 0.0
