"""Pins of the oracle's FIFO history window (Sec. 3.1)."""
from collections import deque

import numpy as np

import oracle


def test_fifo_window_keeps_the_newest_records():
    rng = np.random.default_rng(0)
    cap, d = 7, 32
    bits = np.zeros((cap, d), np.uint16)
    lens = np.full(cap, -1, np.int32)
    total = 0
    window = deque(maxlen=cap)                      # (record id) newest last
    for n in [3, 1, 0, 5, 7, 9, 2, 20]:
        emb = rng.standard_normal((n, d)).astype(np.float32)
        out = np.arange(total, total + n, dtype=np.int32)      # record id as its length
        bits, lens, total = oracle.store_insert(bits, lens, total, emb, out, cap)
        window.extend(range(total - n, total))
        # exactly the newest min(total, cap) records, each in row id mod cap
        assert sorted(int(v) for v in lens if v >= 0) == sorted(window)
        for rid in window:
            assert lens[rid % cap] == rid
        for i in range(n):
            if (total - n + i) in window:
                assert np.array_equal(bits[(total - n + i) % cap], oracle.round_to_bf16(emb[i]))


def test_rows_in_use_are_a_prefix_until_full():
    cap, d = 10, 32
    bits, lens = np.zeros((cap, d), np.uint16), np.full(cap, -1, np.int32)
    bits, lens, total = oracle.store_insert(bits, lens, 0, np.ones((4, d), np.float32), np.arange(4), cap)
    assert total == 4 and list(lens[:4]) == [0, 1, 2, 3] and np.all(lens[4:] == -1)
