"""sage_predict_noalloc: the neighbour search + histogram of sage_predict_layout
with its scratch memory in the library's static device array instead of a
caller workspace. Called through the C ABI and compared bit for bit with
sage_predict_layout on the same inputs, on consecutive calls that shrink (the
array keeps the previous call's contents)."""
import ctypes

import numpy as np
import pytest
import torch

from paper_2603_07917_amd import sage, workloads

pytestmark = pytest.mark.gpu

SAGE_EWORKSPACE = -2
SCRATCH = 64 << 20            # SAGE_NOALLOC_SCRATCH_BYTES


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def host(t):
    torch.cuda.synchronize()
    return t.cpu().numpy()


def outputs(Q, k, B):
    return (torch.full((Q, k), 7, dtype=torch.int32, device="cuda"),
            torch.full((Q, k), 7.0, dtype=torch.float32, device="cuda"),
            torch.full((Q, B), 7, dtype=torch.int32, device="cuda"),
            torch.full((Q, B), 7.0, dtype=torch.float32, device="cuda"))


def noalloc(lib, qb, ql, hb, hl, hist_len, N, d, k, tau, edges, B, out):
    return lib.sage_predict_noalloc(qb.data_ptr(), sage.LAYOUTS[ql], qb.shape[1] if ql == "panels" else qb.shape[0],
                                    hb.data_ptr(), sage.LAYOUTS[hl], hist_len.data_ptr(), N, d, k, float(tau),
                                    edges.data_ptr(), B, *[t.data_ptr() for t in out], sage._stream())


# (Q, N, d, k, B, query layout, store layout): the few-query stream path on a
# large store, then smaller inputs on the stream and filtered paths
CALLS = [(8, 400000, 256, 128, 256, "panels", "panels"),
         (5, 100000, 128, 64, 64, "panels", "rows"),
         (40, 20000, 64, 16, 32, "rows", "panels")]


def test_noalloc_matches_workspace_entry_point():
    lib = sage.load_library()
    for Q, N, d, k, B, ql, hl in CALLS:
        print(f"call Q={Q} N={N} d={d} k={k} B={B} {ql}/{hl}", flush=True)
        need = sage.predict_workspace_bytes(Q, N, d, k, B)
        assert 0 < need <= SCRATCH
        w = workloads.small_predict(Q=Q, N=N, d=d, k=k, B=B, seed=Q + N, clusters=6)
        qb = sage.ingest_bf16(dev(w.queries), ql)
        hb = sage.ingest_bf16(dev(w.hist_emb), hl)
        hist_len, edges = dev(w.hist_len), dev(w.bin_edges)
        ref = [host(t) for t in sage.predict(qb, hb, hist_len, k, 0.8, edges)]
        out = outputs(Q, k, B)
        assert noalloc(lib, qb, ql, hb, hl, hist_len, N, d, k, 0.8, edges, B, out) == 0
        for a, b in zip(ref, [host(t) for t in out]):
            assert np.array_equal(a.view(np.uint8), b.view(np.uint8))


def test_noalloc_rejects_scratch_beyond_the_array():
    lib = sage.load_library()
    Q, N, d, k, B = 4096, 262144, 768, 64, 256
    assert sage.predict_workspace_bytes(Q, N, d, k, B) > SCRATCH
    t = torch.zeros(64, dtype=torch.int32, device="cuda")
    p = t.data_ptr()
    st = lib.sage_predict_noalloc(p, 1, Q, p, 1, p, N, d, k, 0.8, p, B, p, p, p, p, sage._stream())
    assert st == SAGE_EWORKSPACE
    assert b"static" in lib.sage_last_error()
    torch.cuda.synchronize()
    assert int(t.abs().sum().item()) == 0                 # nothing was enqueued
