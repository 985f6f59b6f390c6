"""Pins of the oracle's storage rounding and similarity (CPU only)."""
import os
import struct

import numpy as np
import pytest
import torch

import oracle
from tests import brute

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _golden_bf16():
    rows = []
    for line in open(os.path.join(GOLDEN, "bf16_rounding.txt")):
        if line.startswith("#") or not line.strip():
            continue
        a, b = line.split()[:2]
        rows.append((int(a, 16), int(b, 16)))
    return rows


def test_bf16_golden_cases():
    rows = _golden_bf16()
    x = np.array([r[0] for r in rows], dtype=np.uint32).view(np.float32)
    got = oracle.round_to_bf16(x)
    assert [int(v) for v in got] == [r[1] for r in rows]


def test_bf16_matches_exhaustive_neighbour_choice():
    rng = np.random.default_rng(1)
    # random bit patterns of finite fp32 values in a moderate range, plus exact ties
    u = rng.integers(0x30000000, 0x4F000000, size=3000, dtype=np.uint32)
    u[:1000] = (u[:1000] & 0xFFFF0000) | 0x8000          # exact half-way cases
    u[1000:1100] |= 0x80000000                           # negatives
    x = u.view(np.float32)
    got = oracle.round_to_bf16(x)
    want = [brute.bf16_round_exact(float(v)) for v in x]
    assert [int(g) for g in got] == want


def test_bf16_matches_torch_conversion():
    rng = np.random.default_rng(2)
    x = (rng.standard_normal(20000) * 3).astype(np.float32)
    got = oracle.round_to_bf16(x)
    want = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(got, want)


def test_bf16_value_roundtrip_exact():
    bits = np.arange(0, 0x7F80, 7, dtype=np.uint16)     # finite non-negative patterns
    vals = oracle.bf16_to_f64(bits)
    for b, v in zip(bits[::50], vals[::50]):
        assert brute.bf16_bits_to_fraction(int(b)) == v


def test_similarity_exact_on_tiny_inputs():
    rng = np.random.default_rng(3)
    q = oracle.round_to_bf16(rng.standard_normal((3, 16)).astype(np.float32))
    h = oracle.round_to_bf16(rng.standard_normal((7, 16)).astype(np.float32))
    S = oracle.similarity(q, h)
    for i in range(3):
        for n in range(7):
            assert S[i, n] == float(brute.dot_exact(q[i], h[n]))


def test_similarity_self_and_orthogonal():
    d = 64
    rng = np.random.default_rng(4)
    x = rng.standard_normal((5, d))
    x /= np.linalg.norm(x, axis=1, keepdims=True)
    hb = oracle.round_to_bf16(x.astype(np.float32))
    S = oracle.similarity(hb[2:3], hb)
    # the row itself scores ~1 (bf16 rounding of a unit vector) and ranks first
    # each component moves by at most 2^-9 relative, so |s - 1| <= 2^-8 + 2^-18
    assert abs(S[0, 2] - 1.0) <= 2.0 ** -8 + 2.0 ** -18
    ids, _ = oracle.topk(S, 1)
    assert ids[0, 0] == 2
    # exactly orthogonal bf16 vectors (disjoint supports) score exactly 0
    a = np.zeros((1, d), np.float32); a[0, : d // 2] = 0.125
    b = np.zeros((1, d), np.float32); b[0, d // 2:] = 0.25
    assert oracle.similarity(oracle.round_to_bf16(a), oracle.round_to_bf16(b))[0, 0] == 0.0


def test_search_blocked_equals_unblocked():
    rng = np.random.default_rng(5)
    q = oracle.round_to_bf16(rng.standard_normal((37, 32)).astype(np.float32))
    h = oracle.round_to_bf16(rng.standard_normal((501, 32)).astype(np.float32))
    ids, sims = oracle.search(q, h, 9, block=8, threads=3)
    ids2, sims2 = oracle.topk(oracle.similarity(q, h), 9)
    assert np.array_equal(ids, ids2) and np.array_equal(sims, sims2)
