"""The seeded generators: determinism, shapes and ranges (CPU only)."""
import numpy as np
import pytest

from paper_2603_07917_amd import workloads


def test_deterministic_and_shaped():
    a = workloads.small_predict(Q=10, N=300, d=32, k=4, B=8, seed=1)
    b = workloads.small_predict(Q=10, N=300, d=32, k=4, B=8, seed=1)
    c = workloads.small_predict(Q=10, N=300, d=32, k=4, B=8, seed=2)
    assert np.array_equal(a.hist_emb, b.hist_emb) and np.array_equal(a.queries, b.queries)
    assert not np.array_equal(a.hist_emb, c.hist_emb)
    assert a.hist_emb.shape == (300, 32) and a.hist_emb.dtype == np.float32
    assert np.allclose(np.linalg.norm(a.hist_emb, axis=1), 1.0, atol=1e-6)
    assert a.hist_len.min() >= 1 and a.hist_len.max() <= 4096
    assert np.all(np.diff(a.bin_edges) > 0) and a.bin_edges[0] == 1 and a.bin_edges[-1] == 4096
    assert np.all((a.bin_repr > a.bin_edges[:-1]) & (a.bin_repr < a.bin_edges[1:]))


def test_config1_recipe():
    w = workloads.make_config(1)
    assert w.hist_emb.shape == (8192, 384) and w.queries.shape == (256, 384)
    assert w.prompt_len.min() >= 16 and w.prompt_len.max() <= 2048
    assert w.bin_edges.shape == (129,)
    # within-cluster cosine is high under the RMS-norm reading of the 0.3 spread
    same = w.hist_emb[w.hist_cluster == 0][:50]
    cos = same @ same.T
    assert np.median(cos[np.triu_indices(len(same), 1)]) > 0.85


def test_index_recipe_small():
    w = workloads.small_index(Q=64, B=1024, seed=3)
    assert w.mass.dtype == np.float32 and w.mass.shape == (64, 1024)
    assert np.all(w.mass >= 0) and np.allclose(w.mass.sum(1), 1.0, atol=1e-4)
    assert (w.mass == 0).any()                    # heavy-tailed: many exact zeros
    assert np.all(w.mass[w.mass > 0] >= np.float32(1e-30))
    assert w.prompt_len.min() >= 8 and w.prompt_len.max() <= 32768


def test_noise_and_zipf_options():
    w = workloads.small_predict(Q=200, N=2000, d=16, k=4, B=8, seed=5, clusters=50,
                                noise_frac=0.1, zipf=1.1)
    assert 0.05 < np.mean(w.hist_cluster == -1) < 0.15
    counts = np.bincount(w.hist_cluster[w.hist_cluster >= 0], minlength=50)
    assert counts.max() > 5 * np.median(counts)  # skewed popularity


def test_trace_is_poisson_and_deterministic():
    from scipy.stats import kstest
    spec = workloads.PredictSpec(Q=1, N=1, d=32, clusters=16, mu_range=(3.0, 6.0), s_range=(0.5, 1.0),
                                 L_max=4096, k=1, B=16)
    t = workloads.make_trace(spec, 77, 20000, 8.0)
    gaps = np.diff(np.concatenate([[0.0], t.arrival]))
    assert np.all(gaps >= 0)
    assert gaps.mean() == pytest.approx(1 / 8.0, rel=0.03)
    assert kstest(gaps, "expon", args=(0, 1 / 8.0)).pvalue > 1e-3
    assert t.output_len.min() >= 1 and t.output_len.max() <= 4096
    assert t.queries.shape == (20000, 32) and t.prompt_len.shape == (20000,)
    np.testing.assert_allclose(np.linalg.norm(t.queries, axis=1), 1.0, atol=1e-5)
    t2 = workloads.make_trace(spec, 77, 20000, 8.0)
    assert np.array_equal(t.arrival, t2.arrival) and np.array_equal(t.output_len, t2.output_len)
