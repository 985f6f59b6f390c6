"""Stage parity of the HIP kernels against the oracle, on identical inputs."""
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


def test_native_library_is_the_one_loaded():
    sage.load_library()
    maps = open("/proc/self/maps").read()
    assert sage.library_path() in maps
    hips = {line.split()[-1] for line in maps.splitlines() if "libamdhip64" in line}
    assert len(hips) == 1, hips       # torch and libsage share one HIP runtime


# ---------------------------------------------------------------- ingest
@pytest.mark.parametrize("n", [1, 3, 4, 1001, 1 << 20])
def test_ingest_bit_exact(n):
    rng = np.random.default_rng(n)
    x = (rng.standard_normal(n) * 2).astype(np.float32)
    if n >= 8:
        x[:8] = np.array([0x3F808000, 0x3F818000, 0x3F808001, 0x3F807FFF, 0xBF808000,
                          0xBF818000, 0x3F7FFFFF, 0x80000000], dtype=np.uint32).view(np.float32)
    got = host(sage.ingest_bf16(dev(x)).view(torch.int16)).view(np.uint16)
    assert np.array_equal(got, oracle.round_to_bf16(x))


# ------------------------------------------------------------------ cost
@pytest.mark.parametrize("B", [1, 100, 1024])
def test_cost(B):
    w = workloads.small_index(Q=1000, B=B, seed=B)
    x = host(sage.cost(dev(w.prompt_len), dev(w.bin_repr)))
    want = oracle.cost(w.prompt_len, w.bin_repr)
    assert np.max(np.abs(x - want) / want) <= 1e-7


# ----------------------------------------------------------------- index
@pytest.mark.parametrize("B", [1, 3, 64, 100, 256, 1000, 1024, 4096])
@pytest.mark.parametrize("Q", [1, 777])
def test_index_fused_and_explicit(Q, B):
    w = workloads.small_index(Q=Q, B=B, seed=Q * 7 + B)
    mass = w.mass.copy()
    mass[Q // 2] = 0.0                         # a row with no mass -> +inf
    x = oracle.cost(w.prompt_len, w.bin_repr)
    g, arg = sage.index(dev(mass), dev(w.prompt_len), dev(w.bin_repr), with_argmin=True)
    g, arg = host(g), host(arg)
    G = parity.check_index(g, mass, x)
    assert arg[Q // 2] == -1
    # an explicit fp32 cost support (the exact cost rounded once) gives the index of that support
    x32 = x.astype(np.float32)
    g2 = host(sage.index(dev(mass), cost=dev(x32)))
    parity.check_index(g2, mass, x32.astype(np.float64))
    # argmin: where the oracle's minimum is clear of the runner-up, bins agree
    Gp, ap = oracle.gittins(mass.astype(np.float64), x)
    fin = np.isfinite(Gp)
    assert np.all((arg[fin] >= 0) & (arg[fin] < B))


def test_index_closed_forms():
    B = 256
    _, r = workloads.log_bins(8192, B)
    I = np.array([0, 100, 5000, 17], dtype=np.int32)
    x = oracle.cost(I, r)
    mass = np.zeros((4, B), np.float32)
    mass[0, 10] = 1.0                         # point mass: index = cost of that bin
    mass[1, 200] = 0.25
    mass[2, 3] = 0.5; mass[2, 250] = 0.5      # two-point: min(a/p, mean)
    mass[3, :] = 1.0 / B
    g, arg = sage.index(dev(mass), dev(I), dev(r), with_argmin=True)
    g, arg = host(g), host(arg)
    assert abs(g[0] - x[0, 10]) <= 1e-6 * x[0, 10] and arg[0] == 10
    assert abs(g[1] - x[1, 200]) <= 1e-6 * x[1, 200] and arg[1] == 200
    a, b = x[2, 3], x[2, 250]
    want = min(a / 0.5, 0.5 * a + 0.5 * b)
    assert abs(g[2] - want) <= 1e-6 * want
    mean = x[3].mean()
    assert g[3] <= mean * (1 + 1e-6)


def test_index_config4_full():
    w = workloads.make_config(4)
    x = oracle.cost(w.prompt_len, w.bin_repr)
    g = host(sage.index(dev(w.mass), dev(w.prompt_len), dev(w.bin_repr)))
    parity.check_index(g, w.mass, x)
    g2 = host(sage.index(dev(w.mass), dev(w.prompt_len), dev(w.bin_repr)))
    assert np.array_equal(g.view(np.uint32), g2.view(np.uint32))   # deterministic


# ------------------------------------------------------------------ rank
@pytest.mark.parametrize("Q", [1, 2, 3, 63, 64, 65, 2047, 2048, 2049, 4096, 4097, 5000, 8192, 8193,
                               16383, 16384, 16385, 65536, 131073])
def test_rank_bit_exact(Q):
    rng = np.random.default_rng(Q)
    g = np.round(rng.uniform(0, 50, size=Q)).astype(np.float32)   # many exact ties
    g[rng.random(Q) < 0.05] = np.inf
    g[rng.random(Q) < 0.01] = 0.0
    order = host(sage.rank(dev(g)))
    parity.check_rank(order, g)
    h = rng.lognormal(8, 3, size=Q).astype(np.float32)            # wide dynamic range
    parity.check_rank(host(sage.rank(dev(h))), h)


@pytest.mark.parametrize("Q", [100, 4096, 8000, 16384, 20000])
def test_rank_all_equal_is_identity(Q):
    # every key tied: the stable order is the request order itself
    order = host(sage.rank(dev(np.full(Q, 7.0, dtype=np.float32))))
    assert np.array_equal(order, np.arange(Q, dtype=np.int32))


def test_rank_negative_and_signed_zero():
    g = np.array([3.0, -0.0, 0.0, -1.5, np.inf, -np.inf, 0.0, -0.0, 2.5], dtype=np.float32)
    order = host(sage.rank(dev(g)))
    assert list(order) == list(np.argsort(g, kind="stable"))


# ------------------------------------------------------------- histogram
@pytest.mark.parametrize("k,B,tau", [(1, 1, 0.8), (32, 128, 0.8), (64, 256, 0.8), (100, 37, 0.5),
                                     (256, 1024, 0.9), (64, 4096, 0.8), (64, 256, 1.0)])
def test_histogram_vs_oracle(k, B, tau):
    rng = np.random.default_rng(k * 31 + B)
    N, Q = 5000, 600
    edges, _ = workloads.log_bins(8192, B)
    L = rng.integers(1, 8193, size=N).astype(np.int32)
    ids = np.stack([rng.choice(N, size=k, replace=False) for _ in range(Q)]).astype(np.int32)
    sims = np.sort(rng.uniform(0.6, 1.0, size=(Q, k)).astype(np.float32), axis=1)[:, ::-1].copy()
    ids[:10, k // 2:] = -1                      # fewer valid neighbours than k
    sims[:10, k // 2:] = -np.inf
    sims[10:20] = rng.uniform(0.1, 0.5, size=(10, k)).astype(np.float32)   # all below tau
    counts, mass = sage.histogram(dev(ids), dev(sims), dev(L), tau, dev(edges))
    parity.check_hist(ids, sims, host(counts), host(mass), L, edges, tau)


@pytest.mark.parametrize("k,B,tau", [(64, 256, 0.8), (256, 1024, 0.9), (100, 37, 0.5), (32, 128, 0.8)])
def test_histogram_many_requests_per_wave(k, B, tau):
    """More requests than resident waves: each wave bins several requests in
    turn, with the next requests' lists and lengths in flight."""
    rng = np.random.default_rng(k * 7 + B)
    N, Q = 100000, 20011
    edges, _ = workloads.log_bins(16384, B)
    L = rng.integers(1, 16385, size=N).astype(np.int32)
    ids = rng.integers(0, N, size=(Q, k)).astype(np.int32)
    ids[:, 1] = ids[:, 0]                       # a repeated neighbour id is binned twice
    sims = rng.uniform(0.5, 1.0, size=(Q, k)).astype(np.float32)
    ids[::97, k // 3:] = -1                     # some short lists
    sims[::89] = 0.3                            # some rows below tau
    counts, mass = sage.histogram(dev(ids), dev(sims), dev(L), tau, dev(edges))
    parity.check_hist(ids, sims, host(counts), host(mass), L, edges, tau)


# ------------------------------------------------------- index refresh (attained service)
def test_index_attained_vs_oracle_full_index_workload():
    w = workloads.make_config(4)
    spec = w.spec
    gen = workloads.generated_tokens(4, spec.Q, spec.L_max)
    g = host(sage.index_attained(dev(w.mass), dev(w.prompt_len), dev(w.bin_repr), dev(gen), 200))
    a = oracle.attained_service(w.prompt_len, gen, 200)
    G, _ = oracle.gittins_attained(w.mass.astype(np.float64), oracle.cost(w.prompt_len, w.bin_repr), a)
    inf = np.isinf(G)
    assert np.array_equal(np.isinf(g), inf)
    rel = np.abs(g[~inf].astype(np.float64) - G[~inf]) / np.abs(G[~inf])
    assert rel.max(initial=0.0) <= parity.INDEX_RTOL, rel.max()
    assert (gen > 0).sum() > spec.Q // 3                             # many running rows
    print(f"attained: {int((gen > 0).sum())} running rows, {int(inf.sum())} with no mass left")


@pytest.mark.parametrize("B,levels,bucket", [(256, 41, 200), (100, 5, 1), (1024, 3, 500), (7, 1, 200)])
def test_index_attained_table_matches_per_level_calls(B, levels, bucket):
    """The refresh table equals sage_index_attained called level by level (same
    arithmetic, bit for bit), and level 0 equals the arrival index."""
    rng = np.random.default_rng(B + levels)
    Q = 777
    mass = rng.dirichlet(np.full(B, 0.3), size=Q).astype(np.float32)
    mass[:3] = 0.0                                                # empty rows: +inf everywhere
    plen = rng.integers(8, 4000, size=Q).astype(np.int32)
    edges, r = workloads.log_bins(16384, B)
    md, pd, rd = dev(mass), dev(plen), dev(r)
    table = host(sage.index_attained_table(md, pd, rd, levels, bucket))
    for lv in range(levels):
        g = host(sage.index_attained(md, pd, rd, dev(np.full(Q, lv * bucket, np.int32)), bucket))
        assert np.array_equal(table[lv].view(np.uint32), g.view(np.uint32)), lv
    assert np.array_equal(table[0].view(np.uint32), host(sage.index(md, pd, rd)).view(np.uint32))
    x = oracle.cost(plen, r)
    G, _ = oracle.gittins_attained(mass.astype(np.float64), x,
                                   oracle.attained_service(plen, np.full(Q, (levels - 1) * bucket), bucket))
    inf = np.isinf(G)
    assert np.array_equal(np.isinf(table[-1]), inf)
    rel = np.abs(table[-1][~inf].astype(np.float64) - G[~inf]) / G[~inf]
    assert rel.max(initial=0.0) <= parity.INDEX_RTOL


@pytest.mark.parametrize("B", [7, 64, 256, 1024])
def test_index_attained_zero_is_the_index_and_argmin(B):
    rng = np.random.default_rng(B)
    Q = 300
    mass = rng.dirichlet(np.full(B, 0.3), size=Q).astype(np.float32)
    plen = rng.integers(8, 4000, size=Q).astype(np.int32)
    edges, r = workloads.log_bins(16384, B)
    g0 = host(sage.index(dev(mass), dev(plen), dev(r)))
    ga = host(sage.index_attained(dev(mass), dev(plen), dev(r), dev(np.zeros(Q, np.int32)), 200))
    assert np.array_equal(g0.view(np.uint32), ga.view(np.uint32))
    gen = rng.integers(0, 3000, size=Q).astype(np.int32)
    gen[:5] = 20000                                               # past every support point (L_max 16384)
    for bucket in (1, 200):
        g, arg = sage.index_attained(dev(mass), dev(plen), dev(r), dev(gen), bucket, with_argmin=True)
        g, arg = host(g), host(arg)
        x = oracle.cost(plen, r)
        G, A = oracle.gittins_attained(mass.astype(np.float64), x, oracle.attained_service(plen, gen, bucket))
        inf = np.isinf(G)
        assert np.array_equal(np.isinf(g), inf) and np.all(arg[inf] == -1)
        rel = np.abs(g[~inf].astype(np.float64) - G[~inf]) / G[~inf]
        assert rel.max(initial=0.0) <= parity.INDEX_RTOL
        assert np.all(inf[:5])
        # the argmin attains the minimum (within the tolerance) and lies above the served cost
        a = oracle.attained_service(plen, gen, bucket)
        ok = ~inf
        rows = np.nonzero(ok)[0]
        assert np.all(x[rows, arg[rows]] > a[rows])


# --------------------------------------------------------- the paper's ablation variants
@pytest.mark.parametrize("B", [7, 256, 1024])
@pytest.mark.parametrize("model", ["resource", "output", "overall"])
def test_index_variants_vs_oracle(B, model):
    rng = np.random.default_rng(B + len(model))
    Q = 400
    mass = rng.dirichlet(np.full(B, 0.2), size=Q).astype(np.float32)
    mass[:3] = 0.0                                                 # empty rows
    plen = rng.integers(8, 8000, size=Q).astype(np.int32)
    _, r = workloads.log_bins(32768, B)
    x = oracle.cost_variant(plen, r, model)
    for noise in (0.0, 0.2):
        p = oracle.mix_uniform(mass.astype(np.float64), noise) if noise > 0 else mass.astype(np.float64)
        g = host(sage.index_variant(dev(mass), dev(plen), dev(r), model, "gittins", noise))
        parity.check_index(g, p, x)
        m = host(sage.index_variant(dev(mass), dev(plen), dev(r), model, "mean", noise))
        want = oracle.mean_index(p, x)
        inf = np.isinf(want)
        assert np.array_equal(np.isinf(m), inf)
        rel = np.abs(m[~inf].astype(np.float64) - want[~inf]) / want[~inf]
        assert rel.max() <= parity.INDEX_RTOL
    if model == "resource":                                        # the adopted choice is sage_index
        g0 = host(sage.index(dev(mass), dev(plen), dev(r)))
        g1 = host(sage.index_variant(dev(mass), dev(plen), dev(r)))
        assert np.array_equal(g0.view(np.uint32), g1.view(np.uint32))


@pytest.mark.parametrize("B", [1, 7, 256, 4096])
def test_mix_uniform_vs_oracle(B):
    rng = np.random.default_rng(B + 5)
    Q = 333
    mass = rng.dirichlet(np.full(B, 0.3), size=Q).astype(np.float32) * rng.uniform(0.5, 2.0, (Q, 1)).astype(np.float32)
    mass[:4] = 0.0                                                 # empty rows stay empty
    for w in (0.0, 0.2, 1.0):
        got = host(sage.mix_uniform(dev(mass), w))
        want = oracle.mix_uniform(mass.astype(np.float64), w)
        assert np.all(got[:4] == 0.0)
        err = np.abs(got.astype(np.float64) - want)
        assert np.all(err <= 2.0 ** -23 * np.abs(want) + 1e-30), (w, err.max())
        t = dev(mass)
        sage.mix_uniform(t, w, out=t)                              # in place
        assert np.array_equal(host(t), got)


@pytest.mark.parametrize("k,B,tau", [(32, 128, 0.8), (64, 256, 0.5), (100, 37, 0.8)])
def test_histogram_unweighted_vs_oracle(k, B, tau):
    rng = np.random.default_rng(k + B)
    N, Q = 5000, 300
    edges, _ = workloads.log_bins(8192, B)
    hist_len = rng.integers(1, 8193, size=N).astype(np.int32)
    ids = np.stack([rng.choice(N, size=k, replace=False) for _ in range(Q)]).astype(np.int32)
    ids[:5, k // 2:] = -1
    sims = np.sort(rng.uniform(0.3, 1.0, size=(Q, k)).astype(np.float32), axis=1)[:, ::-1].copy()
    sims[5:10] = 0.2                                               # nobody above tau
    counts, mass = sage.histogram_variant(dev(ids), dev(sims), dev(hist_len), tau, dev(edges), "uniform")
    counts, mass = host(counts), host(mass)
    c, m = oracle.histogram(ids, sims, hist_len, edges, tau, weighting="uniform")
    assert np.array_equal(counts, c)
    assert np.abs(mass.astype(np.float64) - m).max() <= parity.MASS_TOL
    # the similarity weighting through the variant entry point is sage_histogram
    c1, m1 = sage.histogram_variant(dev(ids), dev(sims), dev(hist_len), tau, dev(edges), "similarity")
    c2, m2 = sage.histogram(dev(ids), dev(sims), dev(hist_len), tau, dev(edges))
    assert np.array_equal(host(c1), host(c2)) and np.array_equal(host(m1), host(m2))


# ---------------------------------------------------------- history window (FIFO store)
def test_store_insert_fifo_bit_exact_and_predict():
    rng = np.random.default_rng(17)
    cap, d = 1000, 64
    edges, r = workloads.log_bins(4096, 32)
    ring = sage.RingStore(cap, d, dev(edges), dev(r), k=16, tau=0.8)
    bits = np.zeros((cap, d), np.uint16)
    lens = np.zeros(cap, np.int32)
    total = 0
    w = workloads.small_predict(Q=20, N=4000, d=d, k=16, B=32, seed=3, clusters=5)
    for n in [1, 299, 0, 700, 1, 1500, 333]:
        a = rng.integers(0, 4000 - n) if n < 4000 else 0
        emb, out = w.hist_emb[a:a + n], w.hist_len[a:a + n]
        ring.insert(dev(emb.reshape(n, d)), dev(out))
        bits, lens, total = oracle.store_insert(bits, lens, total, emb.reshape(n, d), out, cap)
        assert ring.total == total and ring.rows == min(total, cap)
        assert np.array_equal(host(ring.ring_emb.view(torch.int16)).view(np.uint16)[:ring.rows], bits[:ring.rows])
        assert np.array_equal(host(ring.ring_len)[:ring.rows], lens[:ring.rows])
    # predictions over the window equal those over the same rows given directly
    q = dev(w.queries)
    a_out = [host(t) for t in ring.predict(q)]
    direct = sage.Store(ring.ring_emb[:ring.rows].clone(), ring.ring_len[:ring.rows].clone(),
                        dev(edges), dev(r), 16, 0.8)
    b_out = [host(t) for t in direct.predict(q)]
    for x, y in zip(a_out, b_out):
        assert np.array_equal(x.view(np.uint8), y.view(np.uint8))
    S = oracle.similarity(oracle.round_to_bf16(w.queries), bits)
    parity.check_topk(a_out[0], a_out[1], S, 16)
