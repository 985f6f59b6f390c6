"""SageSched scheduling-decision path on MI355X (gfx950).

The HIP library is loaded lazily, on first use of one of the entry points,
so that importing ``paper_2603_07917_amd.workloads`` needs no GPU library.
"""
_API = ("ingest_bf16", "predict", "histogram", "cost", "index", "rank", "schedule", "Store",
        "library_path", "load_library", "SageError", "StageTimer", "predict_workspace_bytes",
        "rank_workspace_bytes")


def __getattr__(name):
    if name in _API:
        from . import sage
        return getattr(sage, name)
    raise AttributeError(name)
