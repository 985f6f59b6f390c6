"""The C-ABI library: loads, exports what include/sage.h declares, and rejects
bad arguments before touching a device (CPU only; no compute calls)."""
import ctypes
import math
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "sage.h")
LIB = os.path.join(ROOT, "paper_2603_07917_amd", "libsage.so")

SAGE_OK, SAGE_EINVAL, SAGE_EWORKSPACE = 0, -1, -2


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(sage_[a-z0-9_]+)\s*\(", text)))


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(LIB):
        from paper_2603_07917_amd import build
        build.build()
    lib = ctypes.CDLL(LIB)
    P, I, F, Z = ctypes.c_void_p, ctypes.c_int, ctypes.c_float, ctypes.c_size_t
    lib.sage_predict.argtypes = [P, I, P, P, I, I, I, F, P, I, P, P, P, P, P, Z, P]
    lib.sage_predict_workspace_bytes.argtypes = [I, I, I, I, I]
    lib.sage_predict_workspace_bytes.restype = Z
    lib.sage_rank_workspace_bytes.argtypes = [I]
    lib.sage_rank_workspace_bytes.restype = Z
    lib.sage_index.argtypes = [P, P, P, P, I, I, P, P, P]
    lib.sage_index_attained.argtypes = [P, P, P, P, I, I, I, P, P, P]
    lib.sage_index_variant.argtypes = [P, P, P, I, I, I, I, F, P, P, P]
    lib.sage_histogram_variant.argtypes = [P, P, I, I, P, I, F, P, I, I, P, P, P]
    lib.sage_store_insert.argtypes = [P, P, I, I, ctypes.c_longlong, I, P, P, P]
    lib.sage_mix_uniform.argtypes = [P, I, I, F, P, P]
    lib.sage_rank.argtypes = [P, I, P, P, Z, P]
    lib.sage_cost.argtypes = [P, I, P, I, P, P]
    lib.sage_histogram.argtypes = [P, P, I, I, P, I, F, P, I, P, P, P]
    lib.sage_ingest_bf16.argtypes = [P, Z, P, P]
    lib.sage_ingest_bf16_panels.argtypes = [P, I, I, P, P]
    lib.sage_panels_from_rows.argtypes = [P, I, I, P, P]
    lib.sage_predict_layout.argtypes = [P, I, I, P, I, P, I, I, I, F, P, I, P, P, P, P, P, Z, P]
    lib.sage_index_attained_table.argtypes = [P, P, P, I, I, I, I, P, P]
    lib.sage_queue_admit.argtypes = [P, I, P, P, I, ctypes.c_longlong, I, P, P, P, P]
    lib.sage_queue_dispatch.argtypes = [P, I, P, I, P, P, P]
    lib.sage_status_string.restype = ctypes.c_char_p
    lib.sage_last_error.restype = ctypes.c_char_p
    return lib


def test_header_declares_the_path():
    names = declared_functions()
    for n in ["sage_predict", "sage_cost", "sage_index", "sage_rank", "sage_histogram",
              "sage_ingest_bf16", "sage_predict_workspace_bytes", "sage_rank_workspace_bytes",
              "sage_status_string", "sage_last_error"]:
        assert n in names


def test_every_declared_symbol_is_exported(lib):
    for name in declared_functions():
        assert hasattr(lib, name), name


def test_status_strings(lib):
    for code in [0, -1, -2, -3, -4]:
        assert lib.sage_status_string(code).startswith(b"SAGE_")
    assert b"unknown" in lib.sage_status_string(7)


# Fake, 16-byte aligned addresses: every call below fails validation before
# any device work, so they are never dereferenced.
A = 0x10000


def _predict(lib, Q=4, N=100, d=64, k=8, tau=0.8, B=16, ptrs=None, ws=A, ws_bytes=1 << 30):
    p = ptrs or {}
    g = lambda n: p.get(n, A)
    return lib.sage_predict(g("q"), Q, g("h"), g("l"), N, d, k, tau, g("e"), B, g("ids"), g("sims"),
                            g("c"), g("m"), ws, ws_bytes, None)


@pytest.mark.parametrize("kw", [dict(k=0), dict(k=257), dict(d=33), dict(d=0), dict(B=0),
                                dict(B=4097), dict(tau=0.0), dict(tau=1.5), dict(tau=math.nan),
                                dict(tau=1e-7), dict(N=0), dict(Q=-1)])
def test_predict_rejects_bad_sizes(lib, kw):
    assert _predict(lib, **kw) == SAGE_EINVAL
    assert lib.sage_last_error() != b""


@pytest.mark.parametrize("name", ["q", "h", "l", "e", "ids", "sims", "c", "m"])
def test_predict_rejects_null_and_misaligned(lib, name):
    assert _predict(lib, ptrs={name: None}) == SAGE_EINVAL
    assert _predict(lib, ptrs={name: A + 4}) == SAGE_EINVAL


def test_predict_layout_validation(lib):
    def call(ql=0, hl=0, **kw):
        a = dict(Q=4, N=100, d=64, k=8, tau=0.8, B=16)
        a.update(kw)
        return lib.sage_predict_layout(A, ql, a["Q"], A, hl, A, a["N"], a["d"], a["k"], a["tau"], A, a["B"],
                                       A, A, A, A, A, 1 << 30, None)
    for ql, hl in [(2, 0), (0, 2), (-1, 1), (1, -1)]:
        assert call(ql, hl) == SAGE_EINVAL
        assert b"layout" in lib.sage_last_error()
    assert call(1, 1, d=48) == SAGE_EINVAL
    assert call(1, 1, k=0) == SAGE_EINVAL
    assert call(1, 1, Q=0) == SAGE_OK


def test_panels_ingest_validation(lib):
    for fn in (lib.sage_ingest_bf16_panels, lib.sage_panels_from_rows):
        assert fn(A, -1, 64, A + 0x100000, None) == SAGE_EINVAL
        assert fn(A, 10, 48, A + 0x100000, None) == SAGE_EINVAL
        assert fn(A, 10, 0, A + 0x100000, None) == SAGE_EINVAL
        assert fn(None, 10, 64, A + 0x100000, None) == SAGE_EINVAL
        assert fn(A + 4, 10, 64, A + 0x100000, None) == SAGE_EINVAL
        assert fn(A, 10, 64, A + 8, None) == SAGE_EINVAL          # misaligned
        assert fn(A, 10, 64, A + 16, None) == SAGE_EINVAL         # overlapping
        assert fn(A, 1 << 30, 64, A + 0x100000, None) == SAGE_EINVAL
        assert fn(None, 0, 64, None, None) == SAGE_OK              # nothing to do


def test_index_table_validation(lib):
    fn = lib.sage_index_attained_table
    a = [A + 0x1000 * i for i in range(4)]
    assert fn(a[0], a[1], a[2], 200, 5, -1, 16, a[3], None) == SAGE_EINVAL      # Q
    assert fn(a[0], a[1], a[2], 200, 5, 10, 0, a[3], None) == SAGE_EINVAL       # B
    assert fn(a[0], a[1], a[2], 0, 5, 10, 16, a[3], None) == SAGE_EINVAL        # bucket
    assert fn(a[0], a[1], a[2], 200, 0, 10, 16, a[3], None) == SAGE_EINVAL      # levels
    assert fn(a[0], a[1], a[2], 1 << 20, 1 << 12, 10, 16, a[3], None) == SAGE_EINVAL   # token range
    assert fn(None, a[1], a[2], 200, 5, 10, 16, a[3], None) == SAGE_EINVAL
    assert fn(a[0], a[1] + 4, a[2], 200, 5, 10, 16, a[3], None) == SAGE_EINVAL
    assert fn(None, None, None, 200, 5, 0, 16, None, None) == SAGE_OK           # nothing to do


def test_queue_validation(lib):
    adm, dis = lib.sage_queue_admit, lib.sage_queue_dispatch
    a = [A + 0x1000 * i for i in range(6)]
    assert adm(a[0], -1, a[1], a[2], 16, 0, 10, a[3], a[4], a[5], None) == SAGE_EINVAL
    assert adm(a[0], 8, a[1], a[2], 0, 0, 10, a[3], a[4], a[5], None) == SAGE_EINVAL       # B
    assert adm(a[0], 8, a[1], a[2], 16, 0, 7, a[3], a[4], a[5], None) == SAGE_EINVAL       # slots < batch
    assert adm(a[0], 8, a[1], a[2], 16, -1, 10, a[3], a[4], a[5], None) == SAGE_EINVAL     # next_request
    assert adm(None, 8, a[1], a[2], 16, 0, 10, a[3], a[4], a[5], None) == SAGE_EINVAL
    assert adm(a[0] + 4, 8, a[1], a[2], 16, 0, 10, a[3], a[4], a[5], None) == SAGE_EINVAL
    assert adm(None, 0, None, None, 16, 0, 0, None, None, None, None) == SAGE_OK           # nothing to do
    assert dis(a[0], -1, a[1], 10, a[2], a[3], None) == SAGE_EINVAL
    assert dis(a[0], 8, a[1], 7, a[2], a[3], None) == SAGE_EINVAL
    assert dis(a[0], 8, None, 10, a[2], a[3], None) == SAGE_EINVAL
    assert dis(a[0], 8, a[1], 10, a[2] + 8, a[3], None) == SAGE_EINVAL
    assert dis(None, 0, None, 0, None, None, None) == SAGE_OK


def test_predict_workspace_too_small(lib):
    need = lib.sage_predict_workspace_bytes(4, 100, 64, 8, 16)
    assert need > 0
    assert _predict(lib, ws_bytes=need - 1) == SAGE_EWORKSPACE
    assert _predict(lib, ws=None) == SAGE_EWORKSPACE


def test_predict_q0_is_noop(lib):
    assert _predict(lib, Q=0, ptrs={n: None for n in ["q", "ids", "sims", "c", "m"]}) == SAGE_OK


def test_workspace_sizes(lib):
    assert lib.sage_predict_workspace_bytes(4, 100, 33, 8, 16) == 0
    assert lib.sage_predict_workspace_bytes(0, 100, 64, 8, 16) == 0
    # at least one descending list of >= 64 keys per (query, history chunk)
    w = lib.sage_predict_workspace_bytes(4096, 262144, 768, 64, 256)
    assert w >= 4096 * 64 * 8
    assert lib.sage_predict_workspace_bytes(8, 1000, 64, 200, 16) >= 8 * 256 * 8
    assert lib.sage_rank_workspace_bytes(0) == 0
    assert lib.sage_rank_workspace_bytes(65536) >= 4 * 4 * 65536


def test_index_rank_cost_hist_validation(lib):
    assert lib.sage_index(A, None, None, A, 4, 16, A, None, None) == SAGE_EINVAL
    assert lib.sage_index(A, None, A, A, 4, 0, A, None, None) == SAGE_EINVAL
    assert lib.sage_index(A, None, A, A, 4, 5000, A, None, None) == SAGE_EINVAL
    assert lib.sage_index(None, A, None, None, 4, 16, A, None, None) == SAGE_EINVAL
    assert lib.sage_index(A + 8, A, None, None, 4, 16, A, None, None) == SAGE_EINVAL
    assert lib.sage_index(None, None, None, None, 0, 16, None, None, None) == SAGE_OK
    # sage_index_attained(mass, prompt_len, bin_repr, generated, bucket, Q, B, index, argmin, stream)
    assert lib.sage_index_attained(A, A, A, A, 0, 4, 16, A, None, None) == SAGE_EINVAL      # bucket < 1
    assert lib.sage_index_attained(A, A, A, None, 200, 4, 16, A, None, None) == SAGE_EINVAL
    assert lib.sage_index_attained(A, A, A, A + 4, 200, 4, 16, A, None, None) == SAGE_EINVAL
    assert lib.sage_index_attained(A, A, A, A, 200, 4, 5000, A, None, None) == SAGE_EINVAL
    assert lib.sage_index_attained(None, None, None, None, 200, 0, 16, None, None, None) == SAGE_OK
    # sage_index_variant(mass, prompt_len, bin_repr, Q, B, cost_model, kind, noise, index, argmin, stream)
    assert lib.sage_index_variant(A, A, A, 4, 16, 3, 0, 0.0, A, None, None) == SAGE_EINVAL    # cost model
    assert lib.sage_index_variant(A, A, A, 4, 16, 0, 2, 0.0, A, None, None) == SAGE_EINVAL    # kind
    assert lib.sage_index_variant(A, A, A, 4, 16, 0, 0, 1.0, A, None, None) == SAGE_EINVAL    # noise
    assert lib.sage_index_variant(A, A, A, 4, 16, 0, 0, -0.1, A, None, None) == SAGE_EINVAL
    assert lib.sage_index_variant(A, None, A, 4, 16, 0, 0, 0.2, A, None, None) == SAGE_EINVAL
    assert lib.sage_index_variant(None, None, None, 0, 16, 1, 1, 0.2, None, None, None) == SAGE_OK
    # sage_mix_uniform(mass, Q, B, weight, out, stream)
    assert lib.sage_mix_uniform(A, 4, 16, 1.5, A, None) == SAGE_EINVAL                     # weight
    assert lib.sage_mix_uniform(A, 4, 16, -0.1, A, None) == SAGE_EINVAL
    assert lib.sage_mix_uniform(A, 4, 0, 0.2, A, None) == SAGE_EINVAL                      # B
    assert lib.sage_mix_uniform(A, 4, 16, 0.2, A + 16, None) == SAGE_EINVAL                # overlap
    assert lib.sage_mix_uniform(A, 4, 16, 0.2, None, None) == SAGE_EINVAL
    assert lib.sage_mix_uniform(A + 4, 4, 16, 0.2, A + 4096, None) == SAGE_EINVAL          # alignment
    assert lib.sage_mix_uniform(None, 0, 16, 0.2, None, None) == SAGE_OK
    # sage_histogram_variant(..., weighting, ...)
    assert lib.sage_histogram_variant(A, A, 4, 8, A, 100, 0.8, A, 16, 2, A, A, None) == SAGE_EINVAL
    # sage_store_insert(emb, out_len, n, d, total, capacity, ring_emb, ring_len, stream)
    assert lib.sage_store_insert(A, A, 4, 48, 0, 10, A, A, None) == SAGE_EINVAL       # d % 32
    assert lib.sage_store_insert(A, A, 4, 64, 0, 0, A, A, None) == SAGE_EINVAL        # capacity
    assert lib.sage_store_insert(A, A, 4, 64, -1, 10, A, A, None) == SAGE_EINVAL      # total
    assert lib.sage_store_insert(A, None, 4, 64, 0, 10, A, A, None) == SAGE_EINVAL
    assert lib.sage_store_insert(None, None, 0, 64, 0, 10, None, None, None) == SAGE_OK
    assert lib.sage_rank(A, 10, A, A, 0, None) == SAGE_EWORKSPACE
    assert lib.sage_rank(None, 10, A, A, 1 << 20, None) == SAGE_EINVAL
    assert lib.sage_rank(A, -1, A, A, 1 << 20, None) == SAGE_EINVAL
    assert lib.sage_rank(None, 0, None, None, 0, None) == SAGE_OK
    assert lib.sage_cost(A, 4, None, 16, A, None) == SAGE_EINVAL
    assert lib.sage_cost(A, 4, A, 0, A, None) == SAGE_EINVAL
    assert lib.sage_histogram(A, A, 4, 0, A, 10, 0.8, A, 16, A, A, None) == SAGE_EINVAL
    assert lib.sage_histogram(A, A, 4, 8, A, 0, 0.8, A, 16, A, A, None) == SAGE_EINVAL
    assert lib.sage_histogram(A, A, 4, 8, A, 10, 2.0, A, 16, A, A, None) == SAGE_EINVAL
    assert lib.sage_histogram(A, None, 4, 8, A, 10, 0.8, A, 16, A, A, None) == SAGE_EINVAL
    assert lib.sage_ingest_bf16(None, 10, A, None) == SAGE_EINVAL
    assert lib.sage_ingest_bf16(A, 100, A + 16, None) == SAGE_EINVAL     # overlap
    assert lib.sage_ingest_bf16(None, 0, None, None) == SAGE_OK


def test_check_inputs_and_debug_hook_validation(lib):
    fn = lib.sage_check_inputs
    fn.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int, ctypes.c_void_p, ctypes.c_int,
                   ctypes.c_void_p, ctypes.c_void_p]
    a = [A + 0x1000 * i for i in range(4)]
    assert fn(a[0], a[1], 0, a[2], 4, a[3], None) == SAGE_EINVAL          # B
    assert fn(a[0], a[1], 5000, a[2], 4, a[3], None) == SAGE_EINVAL       # B
    assert fn(a[0], a[1], 16, a[2], -1, a[3], None) == SAGE_EINVAL        # Q
    assert fn(a[0], a[1], 16, a[2], 4, None, None) == SAGE_EINVAL         # status
    assert fn(a[0] + 8, a[1], 16, a[2], 4, a[3], None) == SAGE_EINVAL     # misaligned
    assert fn(a[0], a[1], 16, a[2] + 4, 4, a[3], None) == SAGE_EINVAL
    hook = lib.sage_debug_theta_floor
    hook.argtypes = [ctypes.c_float]
    assert hook(math.nan) == SAGE_EINVAL
    assert hook(-math.inf) == SAGE_OK                                      # off (the default)


def test_panels_ingest_rejects_rows_at_2_pow_29(lib):
    # rows * 4 pieces must fit in int32 inside the kernels
    for fn in (lib.sage_ingest_bf16_panels, lib.sage_panels_from_rows):
        assert fn(A, 1 << 29, 32, A + (1 << 40), None) == SAGE_EINVAL
        assert b"2^29" in lib.sage_last_error()


def test_predict_noalloc_rejects_before_enqueue(lib):
    fn = lib.sage_predict_noalloc
    P, I, F = ctypes.c_void_p, ctypes.c_int, ctypes.c_float
    fn.argtypes = [P, I, I, P, I, P, I, I, I, F, P, I, P, P, P, P, P]
    # a search needing more scratch than the static array: SAGE_EWORKSPACE, before any device call
    assert fn(A, 1, 4096, A, 1, A, 262144, 768, 64, 0.8, A, 256, A, A, A, A, None) == SAGE_EWORKSPACE
    assert b"static" in lib.sage_last_error()
    assert fn(A, 1, 4, A, 1, A, 100, 48, 8, 0.8, A, 16, A, A, A, A, None) == SAGE_EINVAL      # d % 32
    assert fn(A, 1, 4, A, 1, A, 100, 64, 0, 0.8, A, 16, A, A, A, A, None) == SAGE_EINVAL      # k


def test_length_predictor_validation(lib):
    P, I, F, Z = ctypes.c_void_p, ctypes.c_int, ctypes.c_float, ctypes.c_size_t
    bi = lib.sage_length_index
    bi.argtypes = [P, I, I, P, P, P, P, Z, P]
    lib.sage_length_index_workspace_bytes.argtypes = [I]
    lib.sage_length_index_workspace_bytes.restype = Z
    a = [A + 0x1000 * i for i in range(5)]
    assert lib.sage_length_index_workspace_bytes(1000) > 4000
    assert bi(a[0], 0, 100, a[1], a[2], a[3], a[4], 1 << 30, None) == SAGE_EINVAL             # N
    assert bi(a[0], 10, 0, a[1], a[2], a[3], a[4], 1 << 30, None) == SAGE_EINVAL              # max_len
    assert bi(a[0], 10, (1 << 20) + 1, a[1], a[2], a[3], a[4], 1 << 30, None) == SAGE_EINVAL
    assert bi(a[0], 10, 100, None, a[2], a[3], a[4], 1 << 30, None) == SAGE_EINVAL
    assert bi(a[0], 10, 100, a[1], a[2], a[3], a[4], 0, None) == SAGE_EWORKSPACE
    pl = lib.sage_predict_by_length
    pl.argtypes = [P, I, P, P, P, I, P, I, I, F, P, I, P, P, P, P, P]
    ok = lambda **kw: dict(dict(Q=4, max_len=100, N=10, k=8, tau=0.8, B=16), **kw)
    def call(**kw):
        c = ok(**kw)
        return pl(a[0], c["Q"], a[1], a[2], a[3], c["max_len"], a[4], c["N"], c["k"], c["tau"], A, c["B"],
                  A, A, A, A, None)
    for bad in (dict(Q=-1), dict(N=0), dict(k=0), dict(k=257), dict(B=0), dict(max_len=0), dict(tau=0.0)):
        assert call(**bad) == SAGE_EINVAL, bad
    assert call(Q=0) == SAGE_OK
