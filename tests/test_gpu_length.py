"""The semantic-unaware predictor (Sec. 4.3's predictor ablation: neighbours by
input-length similarity) against the oracle: the length index is a stable
sort of the stored lengths; neighbour ids and similarities are bit-exact (both
sides take the choice on the same fp32 quotient, ties to the lower index), so
counts are bit-exact and masses within the histogram's tolerance."""
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


def run(prompt_len, hist_prompt_len, max_len, hist_len, k, tau, edges):
    idx = sage.LengthIndex(dev(hist_prompt_len.astype(np.int32)), max_len)
    out = sage.predict_by_length(dev(prompt_len.astype(np.int32)), idx, dev(hist_len), k, tau, dev(edges))
    return idx, [host(t) for t in out]


def check(prompt_len, hist_prompt_len, max_len, hist_len, k, tau, edges, gpu):
    ids, sims, counts, mass = gpu
    oi, os_, oc, om = oracle.predict_by_length(prompt_len, hist_prompt_len, max_len, hist_len, k, tau, edges)
    assert np.array_equal(ids, oi), "neighbour ids differ"
    assert np.array_equal(sims.astype(np.float64)[oi >= 0], os_[oi >= 0]), "similarities differ"
    assert np.all(np.isneginf(sims[oi < 0]))
    assert np.array_equal(counts, oc), "counts differ"
    assert np.abs(mass.astype(np.float64) - om).max(initial=0.0) <= parity.MASS_TOL


def test_length_index_is_a_stable_sort():
    rng = np.random.default_rng(1)
    L = rng.integers(-3, 600, size=50000).astype(np.int32)      # some below 1 and above max_len
    max_len = 500
    idx = sage.LengthIndex(dev(L), max_len)
    Lc = np.clip(L, 1, max_len)
    want = np.lexsort((np.arange(len(L)), Lc)).astype(np.int32)
    assert np.array_equal(host(idx.by_len), want)
    assert np.array_equal(host(idx.sorted_len), Lc[want])
    off = host(idx.len_off)
    assert np.array_equal(off, np.searchsorted(Lc[want], np.arange(max_len + 2), side="left"))


CASES = [  # (Q, N, k, max_len, seed)
    (300, 20000, 32, 2048, 1),
    (257, 50000, 64, 8192, 2),
    (64, 30000, 128, 4096, 3),
    (40, 10000, 256, 2048, 4),
    (50, 100, 128, 2048, 5),          # N < k: padding
    (70, 5000, 64, 300, 6),           # many records per length (ties across both sides)
]


@pytest.mark.parametrize("Q,N,k,max_len,seed", CASES)
def test_predict_by_length_vs_oracle(Q, N, k, max_len, seed):
    print(f"case Q={Q} N={N} k={k} max_len={max_len}", flush=True)
    rng = np.random.default_rng(seed)
    hist_prompt = np.clip(np.rint(np.exp(rng.normal(6.0, 1.0, N))), 1, 2 * max_len).astype(np.int32)
    prompt = np.clip(np.rint(np.exp(rng.normal(6.0, 1.2, Q))), 0, 4 * max_len).astype(np.int32)
    prompt[:3] = [0, 1, 3 * max_len]                                   # below 1, 1, above max_len
    prompt[3] = hist_prompt[7]                                         # a length that is stored
    hist_len = rng.integers(1, 4097, size=N).astype(np.int32)
    edges, _ = workloads.log_bins(4096, 64)
    _, gpu = run(prompt, hist_prompt, max_len, hist_len, k, 0.8, edges)
    check(prompt, hist_prompt, max_len, hist_len, k, 0.8, edges, gpu)


def test_predict_by_length_equal_ratio_both_sides():
    # I = 100: lengths 80 and 125 share s = 0.8 (and 50 / 200 share 0.5); the
    # k-th neighbour falls inside such a level, so the lower indices win
    # across both sides
    L = np.array([125, 80, 200, 50, 125, 80, 100, 200, 50, 80] * 30, dtype=np.int32)
    hist_len = np.arange(1, len(L) + 1, dtype=np.int32)
    edges, _ = workloads.log_bins(512, 16)
    for k in (1, 30, 31, 45, 100, 200, 256):
        prompt = np.array([100, 100, 99, 101], dtype=np.int32)
        _, gpu = run(prompt, L, 1000, hist_len, k, 0.8, edges)
        check(prompt, L, 1000, hist_len, k, 0.8, edges, gpu)


@pytest.mark.timeout(600)
def test_predict_by_length_mid_workload_sampled():
    """The mid workload's store (262,144 records) and all 4,096 requests; the
    oracle checks a seeded sample of 256 of them."""
    w = workloads.make_config(2)
    spec = w.spec
    idx, gpu = run(w.prompt_len, w.hist_prompt_len, spec.L_max, w.hist_len, spec.k, spec.tau, w.bin_edges)
    rows = np.sort(np.random.default_rng(2).choice(spec.Q, size=256, replace=False))
    check(w.prompt_len[rows], w.hist_prompt_len, spec.L_max, w.hist_len, spec.k, spec.tau, w.bin_edges,
          [a[rows] for a in gpu])
