"""Python binding of libsage (ctypes): argument marshalling only.

Every stage runs in the library's HIP kernels; PyTorch provides device
memory and the current stream. There is no CPU fallback: if the library is
missing or the device is not gfx950, calls raise.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(_HERE, "libsage.so")
_lib = None


class SageError(RuntimeError):
    pass


def library_path() -> str:
    return _LIB_PATH


def load_library():
    """Load libsage.so (after torch, so that both share one HIP runtime)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB_PATH):
        raise SageError(f"{_LIB_PATH} is not built; run `python -m paper_2603_07917_amd.build`")
    lib = ctypes.CDLL(_LIB_PATH)
    P, I, F, Z, S = ctypes.c_void_p, ctypes.c_int, ctypes.c_float, ctypes.c_size_t, ctypes.c_void_p
    sig = {
        "sage_ingest_bf16": (I, [P, Z, P, S]),
        "sage_predict_workspace_bytes": (Z, [I, I, I, I, I]),
        "sage_predict": (I, [P, I, P, P, I, I, I, F, P, I, P, P, P, P, P, Z, S]),
        "sage_predict_layout": (I, [P, I, I, P, I, P, I, I, I, F, P, I, P, P, P, P, P, Z, S]),
        "sage_ingest_bf16_panels": (I, [P, I, I, P, S]),
        "sage_panels_from_rows": (I, [P, I, I, P, S]),
        "sage_histogram": (I, [P, P, I, I, P, I, F, P, I, P, P, S]),
        "sage_cost": (I, [P, I, P, I, P, S]),
        "sage_index": (I, [P, P, P, P, I, I, P, P, S]),
        "sage_index_attained": (I, [P, P, P, P, I, I, I, P, P, S]),
        "sage_index_attained_table": (I, [P, P, P, I, I, I, I, P, S]),
        "sage_index_variant": (I, [P, P, P, I, I, I, I, F, P, P, S]),
        "sage_histogram_variant": (I, [P, P, I, I, P, I, F, P, I, I, P, P, S]),
        "sage_store_insert": (I, [P, P, I, I, ctypes.c_longlong, I, P, P, S]),
        "sage_queue_admit": (I, [P, I, P, P, I, ctypes.c_longlong, I, P, P, P, S]),
        "sage_queue_dispatch": (I, [P, I, P, I, P, P, S]),
        "sage_rank_workspace_bytes": (Z, [I]),
        "sage_rank": (I, [P, I, P, P, Z, S]),
        "sage_simulate": (I, [P, P, P, I, P, I, I, I, I, ctypes.c_double, I, P, P]),
        "sage_mix_uniform": (I, [P, I, I, F, P, S]),
        "sage_check_inputs": (I, [P, P, I, P, I, P, S]),
        "sage_predict_noalloc": (I, [P, I, I, P, I, P, I, I, I, F, P, I, P, P, P, P, S]),
        "sage_predict_stats": (I, [P, Z, I, I, I, I, I, ctypes.POINTER(ctypes.c_longlong), S]),
        "sage_length_index_workspace_bytes": (Z, [I]),
        "sage_length_index": (I, [P, I, I, P, P, P, P, Z, S]),
        "sage_predict_by_length": (I, [P, I, P, P, P, I, P, I, I, F, P, I, P, P, P, P, S]),
        "sage_debug_theta_floor": (I, [F]),
        "sage_status_string": (ctypes.c_char_p, [I]),
        "sage_last_error": (ctypes.c_char_p, []),
        "sage_timer_create": (I, [I, ctypes.POINTER(P)]),
        "sage_timer_destroy": (I, [P]),
        "sage_timer_attach": (I, [P]),
        "sage_timer_only": (I, [P, ctypes.c_char_p]),
        "sage_timer_reset": (I, [P]),
        "sage_timer_count": (I, [P]),
        "sage_timer_get": (I, [P, I, ctypes.POINTER(ctypes.c_char_p), ctypes.POINTER(I),
                               ctypes.POINTER(ctypes.c_double)]),
    }
    for name, (res, args) in sig.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    _lib = lib
    return lib


def _check(status: int):
    if status != 0:
        lib = load_library()
        raise SageError(f"{lib.sage_status_string(status).decode()}: {lib.sage_last_error().decode()}")


def _stream() -> int:
    return torch.cuda.current_stream().cuda_stream


def _ptr(t: Optional[torch.Tensor]):
    return None if t is None else t.data_ptr()


def _dev(t: torch.Tensor, dtype, name: str, ndim: Optional[int] = None) -> torch.Tensor:
    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise SageError(f"{name} must be a CUDA (HIP) tensor")
    if t.dtype != dtype:
        raise SageError(f"{name} must be {dtype}, got {t.dtype}")
    if ndim is not None and t.dim() != ndim:
        raise SageError(f"{name} must have {ndim} dimensions")
    if not t.is_contiguous():
        raise SageError(f"{name} must be contiguous")
    return t


# ------------------------------------------------------------------ stages
# Layouts of an embedding matrix of R rows x d columns: "rows" is a 2-D tensor
# [R, d]; "panels" is a 3-D tensor [d / 32, R, 32] (32-column panels, each
# holding its columns of every row contiguously: the fast layout for search).
LAYOUTS = {"rows": 0, "panels": 1}


def ingest_bf16(x: torch.Tensor, layout: str = "rows") -> torch.Tensor:
    """fp32 embeddings -> bf16 (round to nearest even), on the device; with
    layout="panels", x must be [R, d] and the result is [d / 32, R, 32]."""
    _dev(x, torch.float32, "x")
    if layout == "rows":
        out = torch.empty(x.shape, dtype=torch.bfloat16, device=x.device)
        _check(load_library().sage_ingest_bf16(_ptr(x), x.numel(), _ptr(out), _stream()))
        return out
    if layout != "panels" or x.dim() != 2 or x.shape[1] % 32 != 0:
        raise SageError("panels ingest takes a 2-D [R, d] tensor with d % 32 == 0")
    R, d = x.shape
    out = torch.empty((d // 32, R, 32), dtype=torch.bfloat16, device=x.device)
    _check(load_library().sage_ingest_bf16_panels(_ptr(x), R, d, _ptr(out), _stream()))
    return out


def to_panels(x: torch.Tensor) -> torch.Tensor:
    """bf16 [R, d] row-major -> [d / 32, R, 32] panel-major (bits unchanged)."""
    _dev(x, torch.bfloat16, "x", 2)
    R, d = x.shape
    out = torch.empty((d // 32, R, 32), dtype=torch.bfloat16, device=x.device)
    _check(load_library().sage_panels_from_rows(_ptr(x), R, d, _ptr(out), _stream()))
    return out


def emb_shape(x: torch.Tensor):
    """(rows, d, layout code) of a bf16 embedding matrix in either layout."""
    if x.dim() == 2:
        return x.shape[0], x.shape[1], LAYOUTS["rows"]
    if x.dim() == 3 and x.shape[2] == 32:
        return x.shape[1], x.shape[0] * 32, LAYOUTS["panels"]
    raise SageError("embeddings must be [R, d] (rows) or [d / 32, R, 32] (panels)")


def predict_workspace_bytes(Q: int, N: int, d: int, k: int, B: int) -> int:
    return int(load_library().sage_predict_workspace_bytes(Q, N, d, k, B))


def predict(queries: torch.Tensor, hist_emb: torch.Tensor, hist_len: torch.Tensor, k: int,
            tau: float, bin_edges: torch.Tensor, workspace: Optional[torch.Tensor] = None,
            out=None):
    """Neighbours, per-bin counts and similarity-weighted masses for each query.
    queries and hist_emb may each be row-major [R, d] or panel-major [d / 32, R, 32]."""
    _dev(queries, torch.bfloat16, "queries")
    _dev(hist_emb, torch.bfloat16, "hist_emb")
    _dev(hist_len, torch.int32, "hist_len", 1)
    _dev(bin_edges, torch.float64, "bin_edges", 1)
    Q, d, q_layout = emb_shape(queries)
    N, d_h, h_layout = emb_shape(hist_emb)
    B = bin_edges.shape[0] - 1
    if d_h != d or hist_len.shape[0] != N:
        raise SageError("shape mismatch between queries, hist_emb and hist_len")
    dev = queries.device
    need = predict_workspace_bytes(Q, N, d, k, B)
    if workspace is None or workspace.numel() < need:
        workspace = torch.empty(max(need, 16), dtype=torch.uint8, device=dev)
    if out is None:
        out = (torch.empty((Q, k), dtype=torch.int32, device=dev),
               torch.empty((Q, k), dtype=torch.float32, device=dev),
               torch.empty((Q, B), dtype=torch.int32, device=dev),
               torch.empty((Q, B), dtype=torch.float32, device=dev))
    ids, sims, counts, mass = out
    _check(load_library().sage_predict_layout(
        _ptr(queries), q_layout, Q, _ptr(hist_emb), h_layout, _ptr(hist_len), N, d, k, float(tau),
        _ptr(bin_edges), B, _ptr(ids), _ptr(sims), _ptr(counts), _ptr(mass), _ptr(workspace),
        workspace.numel(), _stream()))
    return ids, sims, counts, mass


def histogram(nbr_ids: torch.Tensor, nbr_sims: torch.Tensor, hist_len: torch.Tensor, tau: float,
              bin_edges: torch.Tensor):
    _dev(nbr_ids, torch.int32, "nbr_ids", 2)
    _dev(nbr_sims, torch.float32, "nbr_sims", 2)
    _dev(hist_len, torch.int32, "hist_len", 1)
    _dev(bin_edges, torch.float64, "bin_edges", 1)
    Q, k = nbr_ids.shape
    B = bin_edges.shape[0] - 1
    counts = torch.empty((Q, B), dtype=torch.int32, device=nbr_ids.device)
    mass = torch.empty((Q, B), dtype=torch.float32, device=nbr_ids.device)
    _check(load_library().sage_histogram(_ptr(nbr_ids), _ptr(nbr_sims), Q, k, _ptr(hist_len),
                                         hist_len.shape[0], float(tau), _ptr(bin_edges), B,
                                         _ptr(counts), _ptr(mass), _stream()))
    return counts, mass


def cost(prompt_len: torch.Tensor, bin_repr: torch.Tensor) -> torch.Tensor:
    _dev(prompt_len, torch.int32, "prompt_len", 1)
    _dev(bin_repr, torch.float64, "bin_repr", 1)
    Q, B = prompt_len.shape[0], bin_repr.shape[0]
    out = torch.empty((Q, B), dtype=torch.float32, device=prompt_len.device)
    _check(load_library().sage_cost(_ptr(prompt_len), Q, _ptr(bin_repr), B, _ptr(out), _stream()))
    return out


def index(mass: torch.Tensor, prompt_len: Optional[torch.Tensor] = None,
          bin_repr: Optional[torch.Tensor] = None, cost: Optional[torch.Tensor] = None,
          with_argmin: bool = False, out: Optional[torch.Tensor] = None):
    """Gittins index per row; the cost is fused in unless `cost` is given."""
    _dev(mass, torch.float32, "mass", 2)
    Q, B = mass.shape
    if cost is not None:
        _dev(cost, torch.float32, "cost", 2)
        if tuple(cost.shape) != (Q, B):
            raise SageError("cost must have the shape of mass")
    else:
        _dev(prompt_len, torch.int32, "prompt_len", 1)
        _dev(bin_repr, torch.float64, "bin_repr", 1)
        if prompt_len.shape[0] != Q or bin_repr.shape[0] != B:
            raise SageError("prompt_len / bin_repr do not match mass")
    g = out if out is not None else torch.empty(Q, dtype=torch.float32, device=mass.device)
    arg = torch.empty(Q, dtype=torch.int32, device=mass.device) if with_argmin else None
    _check(load_library().sage_index(_ptr(mass), _ptr(cost), _ptr(prompt_len), _ptr(bin_repr), Q, B,
                                     _ptr(g), _ptr(arg), _stream()))
    return (g, arg) if with_argmin else g


def index_attained(mass: torch.Tensor, prompt_len: torch.Tensor, bin_repr: torch.Tensor,
                   generated: torch.Tensor, bucket: int = 200, with_argmin: bool = False,
                   out: Optional[torch.Tensor] = None):
    """Index of running requests from their remaining cost (refreshed at bucket boundaries)."""
    _dev(mass, torch.float32, "mass", 2)
    _dev(prompt_len, torch.int32, "prompt_len", 1)
    _dev(bin_repr, torch.float64, "bin_repr", 1)
    _dev(generated, torch.int32, "generated", 1)
    Q, B = mass.shape
    if prompt_len.shape[0] != Q or generated.shape[0] != Q or bin_repr.shape[0] != B:
        raise SageError("prompt_len / generated / bin_repr do not match mass")
    g = out if out is not None else torch.empty(Q, dtype=torch.float32, device=mass.device)
    arg = torch.empty(Q, dtype=torch.int32, device=mass.device) if with_argmin else None
    _check(load_library().sage_index_attained(_ptr(mass), _ptr(prompt_len), _ptr(bin_repr),
                                              _ptr(generated), int(bucket), Q, B, _ptr(g), _ptr(arg),
                                              _stream()))
    return (g, arg) if with_argmin else g


def index_attained_table(mass: torch.Tensor, prompt_len: torch.Tensor, bin_repr: torch.Tensor, levels: int,
                         bucket: int = 200, out: Optional[torch.Tensor] = None):
    """Refresh table: [levels, Q] indices, row lv after lv * bucket generated tokens."""
    _dev(mass, torch.float32, "mass", 2)
    _dev(prompt_len, torch.int32, "prompt_len", 1)
    _dev(bin_repr, torch.float64, "bin_repr", 1)
    Q, B = mass.shape
    if prompt_len.shape[0] != Q or bin_repr.shape[0] != B:
        raise SageError("prompt_len / bin_repr do not match mass")
    g = out if out is not None else torch.empty((levels, Q), dtype=torch.float32, device=mass.device)
    if tuple(g.shape) != (levels, Q) or not g.is_contiguous():
        raise SageError("out must be a contiguous [levels, Q] tensor")
    _check(load_library().sage_index_attained_table(_ptr(mass), _ptr(prompt_len), _ptr(bin_repr), int(bucket),
                                                    int(levels), Q, B, _ptr(g), _stream()))
    return g


COST_MODELS = {"resource": 0, "output": 1, "overall": 2}
INDEX_KINDS = {"gittins": 0, "mean": 1}
WEIGHTINGS = {"similarity": 0, "uniform": 1}


def index_variant(mass: torch.Tensor, prompt_len: torch.Tensor, bin_repr: torch.Tensor,
                  cost_model: str = "resource", kind: str = "gittins", noise: float = 0.0,
                  with_argmin: bool = False, out: Optional[torch.Tensor] = None):
    """The index under the paper's ablation choices (cost model, Gittins or mean, uniform noise)."""
    _dev(mass, torch.float32, "mass", 2)
    _dev(prompt_len, torch.int32, "prompt_len", 1)
    _dev(bin_repr, torch.float64, "bin_repr", 1)
    Q, B = mass.shape
    if prompt_len.shape[0] != Q or bin_repr.shape[0] != B:
        raise SageError("prompt_len / bin_repr do not match mass")
    if cost_model not in COST_MODELS or kind not in INDEX_KINDS:
        raise SageError(f"unknown cost model {cost_model!r} or index kind {kind!r}")
    g = out if out is not None else torch.empty(Q, dtype=torch.float32, device=mass.device)
    arg = torch.empty(Q, dtype=torch.int32, device=mass.device) if with_argmin else None
    _check(load_library().sage_index_variant(_ptr(mass), _ptr(prompt_len), _ptr(bin_repr), Q, B,
                                             COST_MODELS[cost_model], INDEX_KINDS[kind], float(noise),
                                             _ptr(g), _ptr(arg), _stream()))
    return (g, arg) if with_argmin else g


def mix_uniform(mass: torch.Tensor, weight: float = 0.2, out: Optional[torch.Tensor] = None) -> torch.Tensor:
    """Each row merged with the uniform distribution at weight : (1 - weight)
    (0.2 is the paper's 1:4 inaccurate prediction); `out` may be `mass`."""
    _dev(mass, torch.float32, "mass", 2)
    Q, B = mass.shape
    res = out if out is not None else torch.empty_like(mass)
    _dev(res, torch.float32, "out", 2)
    if tuple(res.shape) != (Q, B):
        raise SageError("out must have the shape of mass")
    _check(load_library().sage_mix_uniform(_ptr(mass), Q, B, float(weight), _ptr(res), _stream()))
    return res


def histogram_variant(nbr_ids: torch.Tensor, nbr_sims: torch.Tensor, hist_len: torch.Tensor, tau: float,
                      bin_edges: torch.Tensor, weighting: str = "uniform"):
    """sage_histogram with a choice of neighbour weight ("similarity" or "uniform")."""
    _dev(nbr_ids, torch.int32, "nbr_ids", 2)
    _dev(nbr_sims, torch.float32, "nbr_sims", 2)
    _dev(hist_len, torch.int32, "hist_len", 1)
    _dev(bin_edges, torch.float64, "bin_edges", 1)
    if weighting not in WEIGHTINGS:
        raise SageError(f"unknown weighting {weighting!r}")
    Q, k = nbr_ids.shape
    B = bin_edges.shape[0] - 1
    counts = torch.empty((Q, B), dtype=torch.int32, device=nbr_ids.device)
    mass = torch.empty((Q, B), dtype=torch.float32, device=nbr_ids.device)
    _check(load_library().sage_histogram_variant(_ptr(nbr_ids), _ptr(nbr_sims), Q, k, _ptr(hist_len),
                                                 hist_len.shape[0], float(tau), _ptr(bin_edges), B,
                                                 WEIGHTINGS[weighting], _ptr(counts), _ptr(mass),
                                                 _stream()))
    return counts, mass


def rank_workspace_bytes(Q: int) -> int:
    return int(load_library().sage_rank_workspace_bytes(Q))


def rank(g: torch.Tensor, workspace: Optional[torch.Tensor] = None,
         out: Optional[torch.Tensor] = None) -> torch.Tensor:
    """Stable ascending order of the index (smaller index served first)."""
    _dev(g, torch.float32, "index", 1)
    Q = g.shape[0]
    need = rank_workspace_bytes(Q)
    if workspace is None or workspace.numel() < need:
        workspace = torch.empty(max(need, 16), dtype=torch.uint8, device=g.device)
    order = out if out is not None else torch.empty(Q, dtype=torch.int32, device=g.device)
    _check(load_library().sage_rank(_ptr(g), Q, _ptr(order), _ptr(workspace), workspace.numel(),
                                    _stream()))
    return order


def schedule(mass: torch.Tensor, prompt_len: torch.Tensor, bin_repr: torch.Tensor):
    """Cost -> index -> rank: returns (index, order)."""
    g = index(mass, prompt_len, bin_repr)
    return g, rank(g)


def simulate(arrival, prompt_len, output_len, order, *, rate: float, servers: int = 1,
             queue_cap: int = 1000, bucket: int = 0, levels: int = 1, informed: Optional[int] = None):
    """Replay a request trace against a queue served in `order` (host-side
    sage_simulate). Arguments are host arrays; `informed` (default: all) is
    the number of leading order positions whose entries carry information.
    Returns (finish [R] float64, preemptions [R] int32) as NumPy arrays."""
    import numpy as np
    if any(isinstance(x, torch.Tensor) and x.is_cuda for x in (arrival, prompt_len, output_len, order)):
        raise SageError("simulate takes host arrays")
    a = np.ascontiguousarray(arrival, dtype=np.float64)
    I = np.ascontiguousarray(prompt_len, dtype=np.int32)
    O = np.ascontiguousarray(output_len, dtype=np.int32)
    o = np.ascontiguousarray(order, dtype=np.int32)
    R = a.shape[0]
    if I.shape != (R,) or O.shape != (R,) or o.shape != (int(levels) * R,):
        raise SageError("arrival / prompt_len / output_len / order shapes do not match")
    finish = np.empty(R, dtype=np.float64)
    pre = np.empty(R, dtype=np.int32)
    n_inf = int(levels) * R if informed is None else int(informed)
    _check(load_library().sage_simulate(a.ctypes.data, I.ctypes.data, O.ctypes.data, R, o.ctypes.data,
                                        int(levels), n_inf, int(bucket), int(servers), float(rate),
                                        int(queue_cap), finish.ctypes.data, pre.ctypes.data))
    return finish, pre


def predict_stats(workspace: torch.Tensor, Q: int, N: int, d: int, k: int, B: int) -> dict:
    """What the last predict with this workspace did (sage_predict_stats;
    synchronises the current stream)."""
    out = (ctypes.c_longlong * 5)()
    _check(load_library().sage_predict_stats(workspace.data_ptr(), workspace.numel(), Q, N, d, k, B, out,
                                             _stream()))
    path = {0: "lists", 1: "filtered", 2: "stream"}[int(out[0])]
    return {"path": path, "candidate_keys": int(out[1]), "flagged": int(out[2]),
            "segments_per_query": int(out[3]), "segment_capacity": int(out[4])}


class LengthIndex:
    """The stored records ordered by input length (sage_length_index), for
    the semantic-unaware predictor: record indices sorted by length (ties by
    index), the sorted lengths, and the first sorted position of each length
    0..max_len+1. Lengths are clamped to [1, max_len]."""

    def __init__(self, hist_prompt_len: torch.Tensor, max_len: int):
        _dev(hist_prompt_len, torch.int32, "hist_prompt_len", 1)
        N = hist_prompt_len.shape[0]
        dev = hist_prompt_len.device
        self.max_len = int(max_len)
        self.N = N
        self.by_len = torch.empty(N, dtype=torch.int32, device=dev)
        self.sorted_len = torch.empty(N, dtype=torch.int32, device=dev)
        self.len_off = torch.empty(self.max_len + 2, dtype=torch.int32, device=dev)
        lib = load_library()
        ws = torch.empty(max(16, lib.sage_length_index_workspace_bytes(N)), dtype=torch.uint8, device=dev)
        _check(lib.sage_length_index(hist_prompt_len.data_ptr(), N, self.max_len, self.by_len.data_ptr(),
                                     self.sorted_len.data_ptr(), self.len_off.data_ptr(), ws.data_ptr(),
                                     ws.numel(), _stream()))
        self._ws = ws                                   # alive until the build has run


def predict_by_length(prompt_len: torch.Tensor, index: LengthIndex, hist_len: torch.Tensor, k: int, tau: float,
                      bin_edges: torch.Tensor, out=None):
    """The semantic-unaware predictor (sage_predict_by_length): neighbours by
    input-length similarity min/max, then the same histogram as predict."""
    _dev(prompt_len, torch.int32, "prompt_len", 1)
    _dev(hist_len, torch.int32, "hist_len", 1)
    _dev(bin_edges, torch.float64, "bin_edges", 1)
    Q, B = prompt_len.shape[0], bin_edges.shape[0] - 1
    dev = prompt_len.device
    if out is None:
        out = (torch.empty((Q, k), dtype=torch.int32, device=dev), torch.empty((Q, k), dtype=torch.float32, device=dev),
               torch.empty((Q, B), dtype=torch.int32, device=dev), torch.empty((Q, B), dtype=torch.float32, device=dev))
    ids, sims, counts, mass = out
    _check(load_library().sage_predict_by_length(prompt_len.data_ptr(), Q, index.by_len.data_ptr(),
                                                 index.sorted_len.data_ptr(), index.len_off.data_ptr(),
                                                 index.max_len, hist_len.data_ptr(), index.N, int(k), float(tau),
                                                 bin_edges.data_ptr(), B, ids.data_ptr(), sims.data_ptr(),
                                                 counts.data_ptr(), mass.data_ptr(), _stream()))
    return ids, sims, counts, mass


CHECK_BITS = {1: "bin edges not finite and strictly increasing",
              2: "bin representatives not finite, non-negative and non-decreasing",
              4: "negative prompt length"}


def check_inputs(bin_edges: Optional[torch.Tensor] = None, bin_repr: Optional[torch.Tensor] = None,
                 prompt_len: Optional[torch.Tensor] = None, status: Optional[torch.Tensor] = None,
                 sync: bool = True):
    """Device check of the bin and prompt-length preconditions
    (sage_check_inputs). With `sync`, waits for the result and raises
    SageError naming each failed condition; otherwise returns the int32
    status tensor for the caller to read later."""
    if bin_edges is None and bin_repr is None:
        raise SageError("check_inputs needs bin_edges or bin_repr (they give B)")
    if bin_edges is not None:
        _dev(bin_edges, torch.float64, "bin_edges", 1)
    if bin_repr is not None:
        _dev(bin_repr, torch.float64, "bin_repr", 1)
    B = bin_edges.shape[0] - 1 if bin_edges is not None else bin_repr.shape[0]
    if bin_edges is not None and bin_repr is not None and bin_repr.shape[0] != B:
        raise SageError("bin_repr must have one entry per bin (len(bin_edges) - 1)")
    Q = 0
    if prompt_len is not None:
        _dev(prompt_len, torch.int32, "prompt_len", 1)
        Q = prompt_len.shape[0]
    dev_ = (bin_edges if bin_edges is not None else bin_repr).device
    if status is None:
        status = torch.empty(4, dtype=torch.int32, device=dev_)
    _check(load_library().sage_check_inputs(_ptr(bin_edges), _ptr(bin_repr), B, _ptr(prompt_len), Q,
                                            _ptr(status), _stream()))
    if not sync:
        return status
    bits = int(status[0].item())
    if bits:
        raise SageError("SAGE_EINVAL: " + "; ".join(v for b, v in CHECK_BITS.items() if bits & b))
    return status


def debug_theta_floor(floor: float):
    """Test hook: raise the pre-pass threshold of later predict calls to at
    least `floor` (-inf: off), forcing queries onto the exact fallback."""
    _check(load_library().sage_debug_theta_floor(float(floor)))


class Store:
    """A resident history store plus reusable device workspaces.

    Holds the bf16 embeddings, the recorded output lengths and the bin edges
    on the device, and reuses the predict / rank workspaces across calls so
    that a steady-state decision allocates nothing new. fp32 embeddings
    (store and queries) are ingested in `layout` ("panels" by default: the
    fast one for the search; results are identical).
    """

    def __init__(self, hist_emb: torch.Tensor, hist_len: torch.Tensor, bin_edges: torch.Tensor,
                 bin_repr: torch.Tensor, k: int, tau: float = 0.8, layout: str = "panels"):
        if layout not in LAYOUTS:
            raise SageError(f"unknown layout {layout!r}")
        self.layout = layout
        if hist_emb.dtype == torch.float32:
            hist_emb = ingest_bf16(hist_emb.contiguous(), layout)
        self.hist_emb = hist_emb
        self.hist_len = hist_len
        self.bin_edges = bin_edges
        self.bin_repr = bin_repr
        check_inputs(bin_edges, bin_repr)              # once per store: the bins' order
        self.k = int(k)
        self.tau = float(tau)
        self._ws = torch.empty(16, dtype=torch.uint8, device=hist_emb.device)
        self._rank_ws = torch.empty(16, dtype=torch.uint8, device=hist_emb.device)

    def _workspace(self, Q: int) -> torch.Tensor:
        N, d, _ = emb_shape(self.hist_emb)
        need = predict_workspace_bytes(Q, N, d, self.k, self.bin_edges.shape[0] - 1)
        if self._ws.numel() < need:
            self._ws = torch.empty(need, dtype=torch.uint8, device=self.hist_emb.device)
        return self._ws

    def predict(self, queries: torch.Tensor, out=None):
        if queries.dtype == torch.float32:
            queries = ingest_bf16(queries.contiguous(), self.layout)
        Q = emb_shape(queries)[0]
        return predict(queries, self.hist_emb, self.hist_len, self.k, self.tau, self.bin_edges,
                       workspace=self._workspace(Q), out=out)

    def decide(self, queries: torch.Tensor, prompt_len: torch.Tensor, out=None):
        """One scheduling decision for a batch: predict, cost+index, rank."""
        ids, sims, counts, mass = self.predict(queries, out=None if out is None else out[:4])
        g = index(mass, prompt_len, self.bin_repr, out=None if out is None else out[4])
        Q = g.shape[0]
        need = rank_workspace_bytes(Q)
        if self._rank_ws.numel() < need:
            self._rank_ws = torch.empty(need, dtype=torch.uint8, device=g.device)
        order = rank(g, workspace=self._rank_ws, out=None if out is None else out[5])
        return ids, sims, counts, mass, g, order


def store_insert(emb: torch.Tensor, out_len: torch.Tensor, total: int, ring_emb: torch.Tensor,
                 ring_len: torch.Tensor) -> int:
    """FIFO insert of a batch of served records into a history ring; returns the new total."""
    _dev(emb, torch.float32, "emb", 2)
    _dev(out_len, torch.int32, "out_len", 1)
    _dev(ring_emb, torch.bfloat16, "ring_emb", 2)
    _dev(ring_len, torch.int32, "ring_len", 1)
    n, d = emb.shape
    cap = ring_emb.shape[0]
    if out_len.shape[0] != n or ring_emb.shape[1] != d or ring_len.shape[0] != cap:
        raise SageError("emb / out_len / ring shapes do not match")
    _check(load_library().sage_store_insert(_ptr(emb), _ptr(out_len), n, d, int(total), cap,
                                            _ptr(ring_emb), _ptr(ring_len), _stream()))
    return int(total) + n


class RingStore(Store):
    """A history store kept as a FIFO window of `capacity` records: served
    requests are inserted with `insert`, the oldest is overwritten once the
    window is full, and predictions search the rows in use."""

    def __init__(self, capacity: int, d: int, bin_edges: torch.Tensor, bin_repr: torch.Tensor, k: int,
                 tau: float = 0.8):
        dev = bin_edges.device
        self.ring_emb = torch.zeros((capacity, d), dtype=torch.bfloat16, device=dev)
        self.ring_len = torch.zeros(capacity, dtype=torch.int32, device=dev)
        self.total = 0
        super().__init__(self.ring_emb[:1], self.ring_len[:1], bin_edges, bin_repr, k, tau, layout="rows")

    @property
    def rows(self) -> int:
        return min(self.total, self.ring_emb.shape[0])

    def insert(self, emb: torch.Tensor, out_len: torch.Tensor):
        self.total = store_insert(emb.contiguous(), out_len, self.total, self.ring_emb, self.ring_len)
        self.hist_emb = self.ring_emb[:self.rows]
        self.hist_len = self.ring_len[:self.rows]

    def predict(self, queries: torch.Tensor, out=None):
        if self.total == 0:
            raise SageError("the history window is empty")
        return super().predict(queries, out=out)


class Queue:
    """A standing queue of pending requests, re-ranked at every decision.

    Each slot holds one pending request's length distribution (mass) and
    prompt length. A decision predicts the new arrivals into the slots freed by
    the previous dispatch, re-indexes every slot, ranks them and dispatches the
    first `batch` (smallest index first), whose slots take the next arrivals.
    Buffers are allocated once; the per-decision bookkeeping (slot refills and
    the dispatched ids) runs in the library's queue kernels.
    """

    def __init__(self, store: Store, mass: torch.Tensor, prompt_len: torch.Tensor, batch: int):
        _dev(mass, torch.float32, "mass", 2)
        _dev(prompt_len, torch.int32, "prompt_len", 1)
        n0, B = mass.shape
        dev = mass.device
        self.store = store
        self.batch = int(batch)
        self.slots = n0 + self.batch
        self.mass = torch.zeros((self.slots, B), dtype=torch.float32, device=dev)
        self.mass[:n0] = mass
        self.prompt_len = torch.ones(self.slots, dtype=torch.int32, device=dev)
        self.prompt_len[:n0] = prompt_len
        self.request = torch.full((self.slots,), -1, dtype=torch.int64, device=dev)
        self.request[:n0] = torch.arange(n0, dtype=torch.int64, device=dev)
        self.next_request = n0
        self.free = torch.arange(n0, self.slots, dtype=torch.int64, device=dev)
        self.index = torch.empty(self.slots, dtype=torch.float32, device=dev)
        self.order = torch.empty(self.slots, dtype=torch.int32, device=dev)
        self._rank_ws = torch.empty(max(16, rank_workspace_bytes(self.slots)), dtype=torch.uint8,
                                    device=dev)
        k = store.k
        self._pred = (torch.empty((self.batch, k), dtype=torch.int32, device=dev),
                      torch.empty((self.batch, k), dtype=torch.float32, device=dev),
                      torch.empty((self.batch, B), dtype=torch.int32, device=dev),
                      torch.empty((self.batch, B), dtype=torch.float32, device=dev))
        self.dispatched = torch.empty(self.batch, dtype=torch.int64, device=dev)

    def decide(self, queries: torch.Tensor, prompt_len: torch.Tensor):
        """Admit `batch` new requests, re-rank the queue, dispatch `batch`.

        Returns the predict outputs of the new requests and the request ids
        dispatched (arrival numbers, the first standing request being 0)."""
        if queries.shape[0] != self.batch or prompt_len.shape[0] != self.batch:
            raise SageError(f"a decision admits exactly {self.batch} requests")
        pred = self.store.predict(queries, out=self._pred)
        if prompt_len.data_ptr() % 16 != 0 or not prompt_len.is_contiguous():
            prompt_len = prompt_len.clone()
        _dev(prompt_len, torch.int32, "prompt_len", 1)
        lib = load_library()
        B = self.mass.shape[1]
        _check(lib.sage_queue_admit(_ptr(self.free), self.batch, _ptr(pred[3]), _ptr(prompt_len), B,
                                    self.next_request, self.slots, _ptr(self.mass), _ptr(self.prompt_len),
                                    _ptr(self.request), _stream()))
        self.next_request += self.batch
        index(self.mass, self.prompt_len, self.store.bin_repr, out=self.index)
        rank(self.index, workspace=self._rank_ws, out=self.order)
        _check(lib.sage_queue_dispatch(_ptr(self.order), self.batch, _ptr(self.request), self.slots,
                                       _ptr(self.free), _ptr(self.dispatched), _stream()))
        return pred, self.dispatched


class StageTimer:
    """Per-kernel HIP-event timing of what the library launches while attached:
    every launch, or only those named `only`."""

    def __init__(self, capacity: int = 4096, only: str | None = None):
        lib = load_library()
        h = ctypes.c_void_p()
        _check(lib.sage_timer_create(capacity, ctypes.byref(h)))
        self._h = h
        if only:
            _check(lib.sage_timer_only(h, only.encode()))

    def __enter__(self):
        _check(load_library().sage_timer_attach(self._h))
        return self

    def __exit__(self, *exc):
        load_library().sage_timer_attach(None)
        return False

    def reset(self):
        _check(load_library().sage_timer_reset(self._h))

    def totals(self) -> dict:
        """{kernel name: (launches, total ms)}; synchronise the device first."""
        lib = load_library()
        res = {}
        for i in range(lib.sage_timer_count(self._h)):
            name = ctypes.c_char_p()
            n = ctypes.c_int()
            ms = ctypes.c_double()
            _check(lib.sage_timer_get(self._h, i, ctypes.byref(name), ctypes.byref(n), ctypes.byref(ms)))
            res[name.value.decode()] = (n.value, ms.value)
        return res

    def close(self):
        if self._h:
            load_library().sage_timer_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
