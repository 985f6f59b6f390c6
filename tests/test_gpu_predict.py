"""sage_predict (similarity + top-k + histogram) against the oracle, and the
whole decision path (predict -> cost/index -> rank) on the named workloads."""
import sys

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


def run_predict(w, k, tau=0.8):
    qb = sage.ingest_bf16(dev(w.queries))
    hb = sage.ingest_bf16(dev(w.hist_emb))
    ids, sims, counts, mass = sage.predict(qb, hb, dev(w.hist_len), k, tau, dev(w.bin_edges))
    return host(ids), host(sims), host(counts), host(mass)


def oracle_scores(w, rows=None):
    qb = oracle.round_to_bf16(w.queries if rows is None else w.queries[rows])
    return oracle.similarity(qb, oracle.round_to_bf16(w.hist_emb))


def check_decision(w, rows, ids, sims, counts, mass, g, order, k, tau):
    """Predict, index and rank of the sampled rows against the oracle's own
    results from the same seeded inputs; returns the number of clean rows."""
    S = oracle_scores(w, rows)
    clean, mass_o, delta = parity.check_predict(ids[rows], sims[rows], counts[rows], mass[rows], S,
                                                w.hist_len, w.bin_edges, tau, k)
    x = oracle.cost(w.prompt_len[rows], w.bin_repr)
    parity.check_index_downstream(g[rows], mass_o, x, delta, np.nonzero(clean)[0])
    parity.check_sorted_stably(order, g)
    return int(clean.sum())


# (Q, N, d, k, B): several query tiles with a ragged tail, history chunks and
# 256-row steps with ragged ends, d with a half 64-wide slice, every list length.
CASES = [
    (70, 3000, 64, 8, 16),
    (130, 5000, 96, 32, 128),
    (64, 4096, 384, 64, 64),
    (65, 7777, 128, 100, 256),
    (40, 3001, 32, 200, 64),
    (33, 2500, 64, 256, 1024),
    (5, 300, 64, 1, 7),
    (3, 10, 64, 32, 16),        # N < k: padded with -1 / -inf
    (8, 300000, 64, 128, 512),  # few queries, hundreds of chunk lists: two-level merge
    (8, 200000, 32, 200, 64),
    # few queries (at most 16): the stream search over the store
    (1, 50001, 768, 64, 256),
    (16, 70000, 96, 256, 64),
    (7, 33333, 2048, 100, 128),
    (16, 20000, 64, 1, 16),
    (9, 65536, 32, 64, 32),
    (4, 40000, 2080, 32, 64),   # d above the stream path's limit: the list path
    (17, 30000, 64, 100, 64),   # one query past the stream path: the list path
    (17, 30000, 64, 64, 64),    # ... and the filtered path
    (4, 16384, 64, 128, 32),    # the smallest store with a threshold sample at k = 128: stream path
    (4, 16383, 64, 128, 32),    # one row less: no sample, the list path without a threshold
]


@pytest.mark.parametrize("Q,N,d,k,B", CASES)
def test_predict_small_vs_oracle(Q, N, d, k, B):
    print(f"case Q={Q} N={N} d={d} k={k} B={B}", flush=True)
    w = workloads.small_predict(Q=Q, N=N, d=d, k=k, B=B, seed=Q + N + d + k, clusters=6)
    ids, sims, counts, mass = run_predict(w, k)
    S = oracle_scores(w)
    parity.check_predict(ids, sims, counts, mass, S, w.hist_len, w.bin_edges, 0.8, k)


def test_panels_ingest_bit_exact():
    """The panel-major store holds exactly the row-major bf16 bits, rearranged."""
    rng = np.random.default_rng(7)
    for R, d in [(1, 32), (1000, 96), (4099, 768)]:
        x = dev(rng.standard_normal((R, d)).astype(np.float32))
        rows = sage.ingest_bf16(x)
        pan = sage.ingest_bf16(x, "panels")
        expect = rows.view(R, d // 32, 32).permute(1, 0, 2).contiguous()
        assert tuple(pan.shape) == (d // 32, R, 32)
        assert torch.equal(pan.view(torch.int16), expect.view(torch.int16))
        assert torch.equal(sage.to_panels(rows).view(torch.int16), expect.view(torch.int16))


LAYOUT_CASES = CASES + [(12, 12000, 64, 8, 16)]


@pytest.mark.parametrize("Q,N,d,k,B", LAYOUT_CASES)
def test_predict_panels_identical_to_rows(Q, N, d, k, B):
    """Every search path (filtered, exact lists, two-level merge, fallback)
    gives bit-identical outputs on panel-major and row-major operands."""
    print(f"case Q={Q} N={N} d={d} k={k} B={B}", flush=True)
    w = workloads.small_predict(Q=Q, N=N, d=d, k=k, B=B, seed=Q + N + d + k, clusters=6)
    if (Q, N) == (12, 12000):                      # overflowing candidates: the exact fallback
        w.hist_emb[:6000] = w.hist_emb[6000]
        w.queries[:6] = w.hist_emb[6000]
    qf, hf, hl, be = dev(w.queries), dev(w.hist_emb), dev(w.hist_len), dev(w.bin_edges)
    ref = [host(t) for t in sage.predict(sage.ingest_bf16(qf), sage.ingest_bf16(hf), hl, k, 0.8, be)]
    for ql, hlay in [("panels", "panels"), ("rows", "panels"), ("panels", "rows")]:
        out = sage.predict(sage.ingest_bf16(qf, ql), sage.ingest_bf16(hf, hlay), hl, k, 0.8, be)
        for a, b in zip(ref, [host(t) for t in out]):
            assert np.array_equal(a.view(np.uint8), b.view(np.uint8)), (ql, hlay)


@pytest.mark.parametrize("Q,N,d,k", [(600, 40000, 64, 32), (40, 40000, 64, 32), (600, 40000, 64, 100),
                                     (8, 40000, 64, 100), (16, 40000, 96, 32)])
def test_predict_ignores_workspace_contents(Q, N, d, k):
    """Outputs do not depend on what the workspace held before the call (every
    intermediate, thresholds included, is written before it is read)."""
    w = workloads.small_predict(Q=Q, N=N, d=d, k=k, B=32, seed=Q + k, clusters=6)
    qb, hb = sage.ingest_bf16(dev(w.queries), "panels"), sage.ingest_bf16(dev(w.hist_emb), "panels")
    hl, be = dev(w.hist_len), dev(w.bin_edges)
    need = sage.predict_workspace_bytes(Q, N, d, k, 32)
    outs = []
    for fill in (0x00, 0x7F, 0xFF):
        ws = torch.full((need,), fill, dtype=torch.uint8, device="cuda")
        outs.append([host(t) for t in sage.predict(qb, hb, hl, k, 0.8, be, workspace=ws)])
    for other in outs[1:]:
        for a, b in zip(outs[0], other):
            assert np.array_equal(a.view(np.uint8), b.view(np.uint8))
    S = oracle_scores(w)
    parity.check_predict(*outs[0], S, w.hist_len, w.bin_edges, 0.8, k)


def test_predict_duplicate_rows_lower_id_first():
    # identical history rows score identically in fp32: the lower index must come first
    w = workloads.small_predict(Q=8, N=600, d=64, k=16, B=16, seed=5, clusters=2)
    h = w.hist_emb.copy()
    h[300:340] = h[100]                       # 40 copies of row 100
    w.hist_emb = h
    w.queries[:] = h[100]
    ids, sims, _, _ = run_predict(w, 16)
    S = oracle_scores(w)
    parity.check_topk(ids, sims, S, 16)
    for q in range(8):
        tied = sims[q] == sims[q, 0]
        assert list(ids[q][tied]) == sorted(ids[q][tied])
        assert ids[q, 0] == 100


def test_predict_candidate_overflow_takes_exact_fallback():
    # Half of the store repeats one vector: queries equal to it see thousands of
    # tied scores (far more survivors than the filtered path keeps), which must
    # be answered exactly by the fallback; the other queries take the fast path.
    w = workloads.small_predict(Q=12, N=12000, d=64, k=8, B=16, seed=21, clusters=4)
    h = w.hist_emb.copy()
    h[:6000] = h[6000]
    w.hist_emb = h
    w.queries[:6] = h[6000]
    ids, sims, counts, mass = run_predict(w, 8)
    S = oracle_scores(w)
    assert list(ids[0]) == list(range(8))          # all tied: lowest indices first
    parity.check_predict(ids, sims, counts, mass, S, w.hist_len, w.bin_edges, 0.8, 8)


def test_predict_tau_fallback_and_all_same_length():
    w = workloads.small_predict(Q=20, N=2000, d=64, k=16, B=32, seed=9, clusters=3)
    w.hist_len[:] = 777
    ids, sims, counts, mass = run_predict(w, 16, tau=1.0)      # nobody reaches tau = 1
    b = oracle.bin_of([777], w.bin_edges)[0]
    assert np.all(counts[:, b] == 16) and np.all(mass[:, b] == 1.0)
    parity.check_predict(ids, sims, counts, mass, oracle_scores(w), w.hist_len, w.bin_edges, 1.0, 16)


@pytest.mark.parametrize("Q,k", [(100, 64), (8, 128), (16, 64)])
def test_predict_deterministic(Q, k):
    # candidate positions come from atomics, so their order varies from run to
    # run; the outputs must not
    w = workloads.small_predict(Q=Q, N=60000, d=128, k=k, B=64, seed=11, clusters=16)
    a = run_predict(w, k)
    b = run_predict(w, k)
    for x, y in zip(a, b):
        assert np.array_equal(x.view(np.uint8), y.view(np.uint8))


def test_config1_end_to_end():
    w = workloads.make_config(1)
    spec = w.spec
    store = sage.Store(dev(w.hist_emb), dev(w.hist_len), dev(w.bin_edges), dev(w.bin_repr),
                       spec.k, spec.tau)
    out = store.decide(dev(w.queries), dev(w.prompt_len))
    ids, sims, counts, mass, g, order = [host(t) for t in out]
    clean = check_decision(w, np.arange(spec.Q), ids, sims, counts, mass, g, order, spec.k, spec.tau)
    print(f"config 1: {clean}/{spec.Q} queries compared through the index", flush=True)


def check_decision_blocked(w, rows, out, block):
    """check_decision over `rows` in blocks of queries (bounded score rows),
    the store widened to fp64 once; also the order against the oracle's
    index of the GPU's own masses. Returns the number of clean rows."""
    ids, sims, counts, mass, g, order = out
    spec = w.spec
    hf = oracle.bf16_to_f64(oracle.round_to_bf16(w.hist_emb))
    clean = 0
    for s0 in range(0, len(rows), block):
        r = rows[s0:s0 + block]
        S = oracle.similarity(oracle.round_to_bf16(w.queries[r]), hf)
        c, mass_o, delta = parity.check_predict(ids[r], sims[r], counts[r], mass[r], S, w.hist_len,
                                                w.bin_edges, spec.tau, spec.k)
        x = oracle.cost(w.prompt_len[r], w.bin_repr)
        parity.check_index_downstream(g[r], mass_o, x, delta, np.nonzero(c)[0])
        clean += int(c.sum())
        print(f"  rows {s0}..{s0 + len(r)}: {int(c.sum())} clean", flush=True)
    parity.check_sorted_stably(order, g)
    # cost + index on the GPU's own masses (identical inputs), then the order
    G_o = parity.check_index(g, mass, oracle.cost(w.prompt_len, w.bin_repr))
    parity.check_rank_vs_oracle(order, G_o)
    return clean


def run_decision(w):
    spec = w.spec
    store = sage.Store(dev(w.hist_emb), dev(w.hist_len), dev(w.bin_edges), dev(w.bin_repr),
                       spec.k, spec.tau)
    out = store.decide(dev(w.queries), dev(w.prompt_len))
    return [host(t) for t in out]


@pytest.mark.timeout(900)
def test_config2_full_size_every_query():
    """The mid workload (4,096 queries, 262,144 rows, d = 768) at full size
    in the benchmark's launch configuration; every query checked."""
    w = workloads.make_config(2)
    out = run_decision(w)
    rows = np.arange(w.spec.Q)
    clean = check_decision_blocked(w, rows, out, 512)
    print(f"config 2: {clean}/{len(rows)} queries compared through the index", flush=True)


@pytest.mark.timeout(900)
def test_config3_full_size_sampled():
    """The GEMM-bound workload (16,384 queries, 1M rows, d = 1024, 10% noise
    rows and queries) at full size: a seeded sample of 2,048 queries holding
    every noise query (they exercise the tau fallback), the first and last
    query, and the rest drawn uniformly."""
    w = workloads.make_config(3)
    Q = w.spec.Q
    out = run_decision(w)
    noise_q = np.nonzero(w.query_cluster < 0)[0]
    rng = np.random.default_rng(3)
    rest = np.setdiff1d(np.arange(Q), np.concatenate([noise_q, [0, Q - 1]]))
    n_more = max(0, 2048 - len(noise_q) - 2)
    rows = np.unique(np.concatenate([noise_q, [0, Q - 1], rng.choice(rest, size=n_more, replace=False)]))
    assert len(rows) == max(2048, len(noise_q) + 2) and np.isin(noise_q, rows).all()
    clean = check_decision_blocked(w, rows, out, 256)
    print(f"config 3: {clean}/{len(rows)} sampled queries ({len(noise_q)} noise) compared through the index",
          flush=True)


def test_stream_path_clustered_store():
    """Few queries against a store whose close neighbours sit side by side (a
    FIFO window that received a burst of similar prompts): a workgroup sees
    more candidates of a query than its LDS slots hold, and the rest go to the
    query's candidate array one by one."""
    Q, N, d, k = 4, 60000, 64, 64
    w = workloads.small_predict(Q=Q, N=N, d=d, k=k, B=64, seed=77, clusters=6)
    rng = np.random.default_rng(77)
    for q in range(Q):
        rows = slice(20000 + 1500 * q, 20000 + 1500 * (q + 1))
        near = w.queries[q] + 0.02 * rng.standard_normal((1500, d)).astype(np.float32)
        w.hist_emb[rows] = near / np.linalg.norm(near, axis=1, keepdims=True)
    ids, sims, counts, mass = run_predict(w, k)
    S = oracle_scores(w)
    parity.check_predict(ids, sims, counts, mass, S, w.hist_len, w.bin_edges, 0.8, k)
    assert np.all((ids >= 20000) & (ids < 26000))          # the burst holds every query's neighbours
