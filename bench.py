"""Benchmark of the scheduling-decision path on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--config 3]

A step is one scheduling decision for a batch of pending requests: bf16
ingest of the query embeddings, similarity search + top-k + histogram
(sage_predict_layout on the panel-major store and queries), fused cost +
Gittins index (sage_index) and the queue ranking (sage_rank). Inputs (the history store, the queries, the prompt
lengths) are resident in HBM before the timed region starts. Prints one JSON
line with the whole-job throughput in decisions per second, the roofline of
the dominant kernel (HIP events over the timed region) and the CPU oracle
timed on a bounded sample of the same workload.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

MFMA_BF16_PEAK_TFLOPS = 2500.0     # MI355X dense bf16 MFMA
PANELS = 1                         # SAGE_LAYOUT_PANELS
HBM_PEAK_GBS = 8000.0              # MI355X HBM3E


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--config", default="3", choices=["1", "2", "3", "4", "5", "ttlt"],
                    help="workload: 1 tiny, 2 mid, 3 gemm-bound (default: the largest batch), 4 index-bound, "
                         "5 streaming, ttlt (a Poisson request trace replayed under FCFS / Mean / Gittins)")
    ap.add_argument("--nodes", type=int, default=64, help="ttlt: servers (8 requests/s each)")
    ap.add_argument("--requests", type=int, default=32768, help="ttlt: requests in the trace")
    ap.add_argument("--load", type=float, default=0.9, help="ttlt: offered load per server")
    ap.add_argument("--cpu-seconds", type=float, default=12.0,
                    help="approximate CPU time budget of the oracle baseline sample")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--graph", action="store_true",
                    help="also capture one step in a HIP graph and time its replays (modes 1-4)")
    ap.add_argument("--calibrate-copy", type=int, default=0, metavar="MIB",
                    help="run one plain device copy of this many MiB first (counter calibration)")
    return ap.parse_args()


def read_traffic(kernel: str, workload_key: str, sources=("k_sim_topk.hip", "sage_device.hpp")):
    """HBM bytes per launch from the committed counter summary, if still current.

    The summary records a hash of the kernel sources the counters were taken
    on; after any change to them the figure is stale and None is returned.
    """
    import hashlib
    path = os.path.join(ROOT, "profiles", f"{kernel}_{workload_key}_traffic.txt")
    if not os.path.exists(path):
        return None
    kv = {}
    for line in open(path):
        if ":" in line and not line.startswith("#"):
            k, v = line.split(":", 1)
            kv[k.strip()] = v.strip()
    h = hashlib.sha256()
    for src in sources:
        h.update(open(os.path.join(ROOT, "paper_2603_07917_amd", "csrc", src), "rb").read())
    if kv.get("kernel_source_sha256_16") != h.hexdigest()[:16]:
        return None
    try:
        return float(kv["hbm_bytes_per_launch"])
    except (KeyError, ValueError):
        return None


def stage_rooflines(stages, rows_per_launch: float, d: int, k: int, B: int, search=None):
    """The HBM-bound stages of the decision: algorithmic bytes per launch
    (query ingest 6 B per element; histogram Q(12k + 8B): ids, sims and the
    gathered lengths in, counts and masses out; index Q(4B + 8): masses and
    prompt lengths in, index out; candidate select: 8 B per candidate key and
    4 B per segment count in, a flag and k ids + sims per query out, the key
    count from sage_predict_stats) over the mean launch time from the timer."""
    per = {"ingest_bf16": 6.0 * rows_per_launch * d,
           "hist": rows_per_launch * (12.0 * k + 8.0 * B),
           "index_scan": rows_per_launch * (4.0 * B + 8.0)}
    if search is not None:
        per["topk_select"] = (8.0 * search["candidate_keys"] + 4.0 * rows_per_launch * search["segments_per_query"]
                              + rows_per_launch * (4.0 + 8.0 * k))
    out = {}
    for name, byts in per.items():
        if name not in stages:
            continue
        n, ms = stages[name]
        us = ms / n * 1e3
        gbs = byts / us / 1e3
        out[name] = {"bytes_per_launch": byts, "avg_launch_us": us, "GB_s": gbs,
                     "frac_of_hbm_peak": gbs / HBM_PEAK_GBS}
    return out


def timed_steps(step, steps: int, label: str, sage, torch, capacity: int = 64):
    """Wall time of `steps` calls of step(i), with HIP events recorded only
    around the launches named `label` (the dominant kernel, whose duration the
    roofline needs) so that the timed work is otherwise the untimed one; then
    `steps` more calls with every launch timed, for the per-stage split.
    Returns (elapsed seconds, (launches, ms) of `label`, {stage: (launches, ms)}
    of the second pass)."""
    timer = sage.StageTimer(capacity=capacity * (steps + 1), only=label)
    with timer:
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for i in range(steps):
            step(i)
        torch.cuda.synchronize()
        elapsed = time.perf_counter() - t0
    dominant = timer.totals()[label]
    timer.close()
    split = sage.StageTimer(capacity=capacity * (steps + 1))
    with split:
        for i in range(steps):
            step(steps + i)
        torch.cuda.synchronize()
    stages = split.totals()
    split.close()
    return elapsed, dominant, stages


def graph_replay(step, steps: int, rows: int, torch) -> dict:
    """One step captured in a HIP graph (every launch on the capturing stream),
    then `steps` replays timed on the wall clock: what a serving loop that
    replays the decision pays per batch."""
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        step()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        step()
    for _ in range(3):
        graph.replay()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(steps):
        graph.replay()
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    return {"ms_per_step": 1e3 * elapsed / steps, "value": rows * steps / elapsed}


def kernel_name(k: int, Q: int = 1 << 30) -> str:
    """The kernel behind the `sim_topk` timer label: the stream search for at
    most 16 queries (large stores), else the filtered path for k <= 64."""
    if Q <= 16:
        return "sim_stream_kernel"
    return "sim_filter_kernel" if k <= 64 else "sim_topk_kernel"


def oracle_threads() -> int:
    return int(os.environ.get("OMP_NUM_THREADS", os.cpu_count() or 1))


def cpu_baseline(w, budget_s: float):
    """The oracle (as it stands) on a bounded sample of the same batch."""
    import oracle
    threads = oracle_threads()
    spec = w.spec
    # the resident store, rounded and widened once: not timed, as on the GPU
    hb = oracle.bf16_to_f64(oracle.round_to_bf16(w.hist_emb))
    block = 128
    done = 0
    t_total = 0.0
    while done < spec.Q and t_total < budget_s:
        rows = slice(done, min(spec.Q, done + block))
        t0 = time.perf_counter()
        qb = oracle.round_to_bf16(w.queries[rows])
        ids, sims = oracle.search(qb, hb, spec.k, block=block, threads=threads)
        counts, mass = oracle.histogram(ids, sims, w.hist_len, w.bin_edges, spec.tau)
        G, arg, order = oracle.schedule(mass, w.prompt_len[rows], w.bin_repr)
        t_total += time.perf_counter() - t0
        done = rows.stop
    return {"value": done / t_total, "unit": "decisions/s", "cores": threads, "kind": "oracle",
            "sample": f"first {done} of the {spec.Q} requests of one batch (full history), "
                      f"{t_total:.1f} s of CPU time; ranking within the sample"}


def cpu_baseline_index(w, budget_s: float):
    """The oracle's cost + Gittins index + rank on blocks of the index-bound
    batch until about budget_s of CPU time."""
    import oracle
    spec = w.spec
    block = 4096
    done, t_total = 0, 0.0
    while done < spec.Q and t_total < budget_s:
        rows = slice(done, min(spec.Q, done + block))
        t0 = time.perf_counter()
        oracle.schedule(w.mass[rows], w.prompt_len[rows], w.bin_repr)
        t_total += time.perf_counter() - t0
        done = rows.stop
    return {"value": done / t_total, "unit": "decisions/s", "cores": oracle_threads(), "kind": "oracle",
            "sample": f"first {done} of the {spec.Q} requests ({spec.B} bins each), blocks of {block}, "
                      f"{t_total:.1f} s of CPU time; ranking within each block"}


def cpu_baseline_streaming(w, standing: int, batch: int, budget_s: float):
    """The oracle's work per streaming decision on the first calls: search +
    histogram of the call's arrivals against the whole store, then cost +
    Gittins index + rank of a standing queue of standing + batch rows, until
    about budget_s of CPU time."""
    import oracle
    spec = w.spec
    hb = oracle.bf16_to_f64(oracle.round_to_bf16(w.hist_emb))     # resident store, untimed
    threads = oracle_threads()
    n_calls = spec.Q // batch
    calls, t_total = 0, 0.0
    plen_queue = np.resize(w.prompt_len, standing + batch)
    while calls < n_calls and t_total < budget_s:
        a = calls * batch
        t0 = time.perf_counter()
        qb = oracle.round_to_bf16(w.queries[a:a + batch])
        ids, sims = oracle.search(qb, hb, spec.k, block=batch, threads=threads)
        _, mass = oracle.histogram(ids, sims, w.hist_len, w.bin_edges, spec.tau)
        queue_mass = np.resize(mass, (standing + batch, spec.B))
        oracle.schedule(queue_mass, plen_queue, w.bin_repr)
        t_total += time.perf_counter() - t0
        calls += 1
    return {"value": calls * batch / t_total, "unit": "decisions/s", "cores": threads, "kind": "oracle",
            "sample": f"first {calls} of the {n_calls} decisions: each searches its {batch} arrivals against "
                      f"all {spec.N} rows, then costs, indexes and ranks a queue of {standing + batch} rows "
                      f"(masses: the call's own predictions repeated, values do not change the work); "
                      f"{t_total:.1f} s of CPU time"}


def main():
    args = parse()
    if args.gpus != 1:
        print(json.dumps({"error": "this build runs on one GPU only; --gpus must be 1",
                          "n_gpus": args.gpus}))
        sys.exit(2)

    import torch
    from paper_2603_07917_amd import sage, workloads

    torch.cuda.set_device(0)
    if args.calibrate_copy:
        n = args.calibrate_copy * (1 << 20) // 4
        a = torch.ones(n, dtype=torch.float32, device="cuda")
        b = torch.empty_like(a)
        b.copy_(a)
        torch.cuda.synchronize()
        del a, b
    if args.config == "ttlt":
        return run_ttlt(args, torch, sage, workloads)
    args.config = int(args.config)
    if args.config == 5:
        return run_streaming(args, torch, sage, workloads)
    if args.config == 4:
        return run_index_bound(args, torch, sage, workloads)
    w = workloads.make_config(args.config)
    spec = w.spec
    Q, N, d, k, B = spec.Q, spec.N, spec.d, spec.k, spec.B
    dev = lambda a: torch.from_numpy(np.ascontiguousarray(a)).cuda()

    # Resident inputs (untimed): history store ingested to bf16 once.
    hist_f32 = dev(w.hist_emb)
    hist = sage.ingest_bf16(hist_f32, "panels")          # panel-major resident store
    del hist_f32
    hist_len = dev(w.hist_len)
    edges = dev(w.bin_edges)
    repr_ = dev(w.bin_repr)
    queries_f32 = dev(w.queries)
    prompt_len = dev(w.prompt_len)

    # Preallocated outputs and workspaces: a step allocates nothing.
    qb = torch.empty((d // 32, Q, 32), dtype=torch.bfloat16, device="cuda")
    ids = torch.empty((Q, k), dtype=torch.int32, device="cuda")
    sims = torch.empty((Q, k), dtype=torch.float32, device="cuda")
    counts = torch.empty((Q, B), dtype=torch.int32, device="cuda")
    mass = torch.empty((Q, B), dtype=torch.float32, device="cuda")
    g = torch.empty(Q, dtype=torch.float32, device="cuda")
    order = torch.empty(Q, dtype=torch.int32, device="cuda")
    ws = torch.empty(max(16, sage.predict_workspace_bytes(Q, N, d, k, B)), dtype=torch.uint8, device="cuda")
    rws = torch.empty(max(16, sage.rank_workspace_bytes(Q)), dtype=torch.uint8, device="cuda")
    lib = sage.load_library()

    def step():
        stream = torch.cuda.current_stream().cuda_stream
        sage._check(lib.sage_ingest_bf16_panels(queries_f32.data_ptr(), Q, d, qb.data_ptr(), stream))
        sage._check(lib.sage_predict_layout(qb.data_ptr(), PANELS, Q, hist.data_ptr(), PANELS,
                                            hist_len.data_ptr(), N, d, k, float(spec.tau),
                                            edges.data_ptr(), B, ids.data_ptr(), sims.data_ptr(),
                                            counts.data_ptr(), mass.data_ptr(), ws.data_ptr(),
                                            ws.numel(), stream))
        sage._check(lib.sage_index(mass.data_ptr(), None, prompt_len.data_ptr(), repr_.data_ptr(), Q,
                                   B, g.data_ptr(), None, stream))
        sage._check(lib.sage_rank(g.data_ptr(), Q, order.data_ptr(), rws.data_ptr(), rws.numel(),
                                  stream))

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()

    elapsed, (n_launch, k1_ms), stages = timed_steps(lambda i: step(), args.steps, "sim_topk", sage, torch)
    print(f"# step: {1e3 * elapsed / args.steps:.3f} ms", file=sys.stderr, flush=True)
    search = sage.predict_stats(ws, Q, N, d, k, B)      # the last step's search (same inputs); synchronises

    ms_per_step = 1e3 * elapsed / args.steps
    value = Q * args.steps / elapsed
    k1_avg_s = k1_ms / n_launch / 1e3
    flops = 2.0 * Q * N * d
    achieved = flops / k1_avg_s / 1e12
    workload_key = workloads.WORKLOAD_NAMES[args.config].split(":")[0]
    traffic = read_traffic("sim_topk", workload_key)

    line = {
        "metric": "scheduling decisions/sec (predict+cost+index+rank)",
        "value": value,
        "unit": "decisions/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": workloads.WORKLOAD_NAMES[args.config], "Q": Q, "N": N, "d": d,
                   "k": k, "B": B, "tau": spec.tau, "layout": "panels", "seed": w.seed},
        "roofline": {"bound": "mfma", "kernel": kernel_name(k), "achieved": achieved,
                     "peak": MFMA_BF16_PEAK_TFLOPS, "unit": "TFLOP/s",
                     "frac": achieved / MFMA_BF16_PEAK_TFLOPS, "traffic": traffic,
                     "avg_launch_us": k1_avg_s * 1e6, "flops_per_launch": flops},
        "stages_us_per_step": {name: 1e3 * ms / args.steps for name, (n, ms) in stages.items()},
        "stage_rooflines": stage_rooflines(stages, Q, d, k, B, search),
        "search": search,
    }
    # measured HBM bytes per launch of the stage kernels, where a current counter summary exists
    for stage, kern, srcs in (("hist", "hist_kernel", ("k_hist.hip", "sage_device.hpp")),
                              ("topk_select", "select_kernel", ("k_sim_topk.hip", "sage_device.hpp"))):
        if stage in line["stage_rooflines"]:
            line["stage_rooflines"][stage]["traffic"] = read_traffic(kern, workload_key, srcs)
    if args.graph:
        line["graph_replay"] = graph_replay(step, args.steps, Q, torch)
    if not args.no_cpu_baseline:
        line["cpu_baseline"] = cpu_baseline(w, args.cpu_seconds)
    print(json.dumps(line), flush=True)


def run_index_bound(args, torch, sage, workloads):
    """The index-bound workload: 65,536 requests that already carry a
    1,024-bin length distribution; a step is cost + Gittins index + rank."""
    w = workloads.make_config(4)
    spec = w.spec
    Q, B = spec.Q, spec.B
    dev = lambda a: torch.from_numpy(np.ascontiguousarray(a)).cuda()
    mass, plen, repr_ = dev(w.mass), dev(w.prompt_len), dev(w.bin_repr)
    g = torch.empty(Q, dtype=torch.float32, device="cuda")
    order = torch.empty(Q, dtype=torch.int32, device="cuda")
    rws = torch.empty(max(16, sage.rank_workspace_bytes(Q)), dtype=torch.uint8, device="cuda")

    def step():
        sage.index(mass, plen, repr_, out=g)
        sage.rank(g, workspace=rws, out=order)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    elapsed, (n_launch, k_ms), stages = timed_steps(lambda i: step(), args.steps, "index_scan", sage, torch)
    avg_s = k_ms / n_launch / 1e3
    k_bytes = Q * (4.0 * B + 8.0)               # masses + prompt lengths in, index out
    achieved = k_bytes / avg_s / 1e9

    # The refresh of running requests (attained service, bucket 200) on the same rows.
    gen = dev(workloads.generated_tokens(4, Q, spec.L_max))
    for _ in range(args.warmup):
        sage.index_attained(mass, plen, repr_, gen, 200, out=g)
    torch.cuda.synchronize()
    timer = sage.StageTimer(capacity=64 * (args.steps + 1))
    with timer:
        for _ in range(args.steps):
            sage.index_attained(mass, plen, repr_, gen, 200, out=g)
        torch.cuda.synchronize()
    n_att, att_ms = timer.totals()["index_attained"]
    timer.close()
    att_s = att_ms / n_att / 1e3
    att_bytes = Q * (4.0 * B + 12.0)
    line = {
        "metric": "scheduling decisions/sec (cost+index+rank)",
        "value": Q * args.steps / elapsed,
        "unit": "decisions/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": 1e3 * elapsed / args.steps,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f64",
        "data": "synthetic",
        "config": {"workload": workloads.WORKLOAD_NAMES[4], "Q": Q, "B": B, "alpha": spec.alpha,
                   "seed": w.seed},
        "roofline": {"bound": "hbm", "kernel": "index_kernel", "achieved": achieved,
                     "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": achieved / HBM_PEAK_GBS,
                     "traffic": read_traffic("index_kernel", "index-bound",
                                             ("k_index_rank.hip", "sage_device.hpp")),
                     "avg_launch_us": avg_s * 1e6, "bytes_per_launch": k_bytes},
        "stages_us_per_step": {name: 1e3 * ms / args.steps for name, (n, ms) in stages.items()},
        "attained_refresh": {"kernel": "index_kernel (attained)", "bucket": 200,
                             "running_rows": int((gen > 0).sum().item()), "avg_launch_us": att_s * 1e6,
                             "achieved_GBs": att_bytes / att_s / 1e9,
                             "frac_of_hbm_peak": att_bytes / att_s / 1e9 / HBM_PEAK_GBS},
    }
    if args.graph:
        line["graph_replay"] = graph_replay(step, args.steps, Q, torch)
    if not args.no_cpu_baseline:
        line["cpu_baseline"] = cpu_baseline_index(w, args.cpu_seconds)
    print(json.dumps(line), flush=True)


def run_streaming(args, torch, sage, workloads):
    """The streaming workload: each call admits 8 new requests (predicted
    against the 4M-row store), re-indexes the 8,200 queued requests, ranks them
    and dispatches 8, so the standing queue stays at 8,192."""
    def log(msg):
        print(f"# {msg}", file=sys.stderr, flush=True)
    spec = workloads.CONFIGS[5]
    batch, standing = 8, 8192
    log("generating the streaming workload")
    w = workloads.make_config(5)
    sq, splen = workloads.make_standing(spec, 5, standing)
    dev = lambda a: torch.from_numpy(np.ascontiguousarray(a)).cuda()
    log("ingesting the store")
    store = sage.Store(dev(w.hist_emb), dev(w.hist_len), dev(w.bin_edges), dev(w.bin_repr), spec.k,
                       spec.tau)
    torch.cuda.empty_cache()
    log("predicting the standing queue")
    _, _, _, smass = store.predict(dev(sq))
    queue = sage.Queue(store, smass.clone(), dev(splen), batch)
    arrivals = dev(w.queries)
    plens = dev(w.prompt_len)
    n_arrivals = arrivals.shape[0] // batch

    def call(c):
        a = (c % n_arrivals) * batch
        queue.decide(arrivals[a:a + batch], plens[a:a + batch])

    for c in range(args.warmup):
        call(c)
    torch.cuda.synchronize()
    log("timed calls")
    starts = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps)]
    ends = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps)]
    def timed_call(i):
        if i < args.steps:
            starts[i].record()
            call(args.warmup + i)
            ends[i].record()
        else:
            call(args.warmup + i)

    elapsed, (n_launch, k1_ms), stages = timed_steps(timed_call, args.steps, "sim_topk", sage, torch)
    lat = np.array([s.elapsed_time(e) for s, e in zip(starts, ends)])
    k1_avg_s = k1_ms / n_launch / 1e3
    k1_bytes = 2.0 * spec.N * spec.d + 2.0 * batch * spec.d
    achieved = k1_bytes / k1_avg_s / 1e9
    line = {
        "metric": "scheduling decisions/sec (predict+cost+index+rank)",
        "value": batch * args.steps / elapsed,
        "unit": "decisions/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": 1e3 * elapsed / args.steps,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": workloads.WORKLOAD_NAMES[5], "calls": args.steps, "batch": batch,
                   "standing": standing, "N": spec.N, "d": spec.d, "k": spec.k, "B": spec.B,
                   "tau": spec.tau, "seed": [workloads.SEED_BASE, 5]},
        "latency_ms": {"p50": float(np.percentile(lat, 50)), "p99": float(np.percentile(lat, 99))},
        "reindexed_rows_per_s": queue.slots * args.steps / elapsed,
        "roofline": {"bound": "hbm", "kernel": kernel_name(spec.k, batch), "achieved": achieved,
                     "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": achieved / HBM_PEAK_GBS,
                     "traffic": read_traffic("sim_stream_kernel", "streaming",
                                             sources=("k_sim_stream.hip", "sage_device.hpp")), "avg_launch_us": k1_avg_s * 1e6, "bytes_per_launch": k1_bytes},
        "stages_us_per_step": {name: 1e3 * ms / args.steps for name, (n, ms) in stages.items()},
    }
    if not args.no_cpu_baseline:
        log("cpu baseline")
        line["cpu_baseline"] = cpu_baseline_streaming(w, standing, batch, args.cpu_seconds)
    print(json.dumps(line), flush=True)


def run_ttlt(args, torch, sage, workloads):
    """A Poisson request trace over the mid workload's history store, replayed
    under each queue order. A step is the trace's whole GPU pass: predict
    every request, then each policy's index values (the refreshed Gittins
    table: one attained-service launch per bucket level) and their rank. The
    host replay (sage_simulate) is timed apart."""
    from paper_2603_07917_amd import simulator

    def log(msg):
        print(f"# {msg}", file=sys.stderr, flush=True)
    spec = workloads.CONFIGS[2]
    R, nodes, bucket, cap = args.requests, args.nodes, 200, 1000
    rps = 8.0 * nodes
    log("generating the store and the trace")
    w = workloads.make_config(2)
    tr = workloads.make_trace(spec, 2, R, rps)
    dev = lambda a: torch.from_numpy(np.ascontiguousarray(a)).cuda()
    store = sage.Store(dev(w.hist_emb), dev(w.hist_len), dev(w.bin_edges), dev(w.bin_repr), spec.k,
                       spec.tau)
    queries, plen = dev(tr.queries), dev(tr.prompt_len)
    rate = simulator.rate_for_load(tr.prompt_len, tr.output_len, rps, nodes, args.load)
    chunk = 16384
    B = spec.B
    mass = torch.empty((R, B), dtype=torch.float32, device="cuda")
    n = min(R, chunk)
    pred_out = (torch.empty((n, spec.k), dtype=torch.int32, device="cuda"),
                torch.empty((n, spec.k), dtype=torch.float32, device="cuda"),
                torch.empty((n, B), dtype=torch.int32, device="cuda"))
    L = simulator.refresh_levels(tr.output_len, bucket)
    table = torch.empty((L, R), dtype=torch.float32, device="cuda")
    g_static = torch.empty(R, dtype=torch.float32, device="cuda")
    g_mean = torch.empty(R, dtype=torch.float32, device="cuda")
    arr32 = dev(tr.arrival.astype(np.float32))
    orders = {"fcfs": torch.empty(R, dtype=torch.int32, device="cuda"),
              "mean": torch.empty(R, dtype=torch.int32, device="cuda"),
              "gittins-static": torch.empty(R, dtype=torch.int32, device="cuda"),
              "gittins": torch.empty(L * R, dtype=torch.int32, device="cuda")}
    rws = torch.empty(max(16, sage.rank_workspace_bytes(L * R)), dtype=torch.uint8, device="cuda")

    def step():
        for s in range(0, R, chunk):
            e = min(R, s + chunk)
            store.predict(queries[s:e], out=tuple(t[:e - s] for t in pred_out) + (mass[s:e],))
        sage.rank(arr32, workspace=rws, out=orders["fcfs"])
        sage.index_variant(mass, plen, store.bin_repr, kind="mean", out=g_mean)
        sage.rank(g_mean, workspace=rws, out=orders["mean"])
        sage.index(mass, plen, store.bin_repr, out=g_static)
        sage.rank(g_static, workspace=rws, out=orders["gittins-static"])
        sage.index_attained_table(mass, plen, store.bin_repr, L, bucket, out=table)
        sage.rank(table.view(-1), workspace=rws, out=orders["gittins"])

    log("warmup")
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    log("timed passes")
    elapsed, (n_launch, k1_ms), stages = timed_steps(lambda i: step(), args.steps, "sim_topk", sage, torch,
                                                     capacity=L + 64)

    log("replaying the trace")
    informed = int(np.isfinite(table.cpu().numpy()).sum())
    host_orders = {pol: (o.cpu().numpy(), L if pol == "gittins" else 1,
                         informed if pol == "gittins" else R, pol == "gittins")
                   for pol, o in orders.items()}
    # The other reading of a refresh that finds no predicted mass above the
    # service received: the request ranks last (+inf) instead of keeping its
    # last index (every entry of the table counts as informed).
    host_orders["gittins (exhausted last)"] = (host_orders["gittins"][0], L, L * R, True)
    # The same policies on inaccurate predictions (Sec. 4.3: a uniform
    # distribution merged in at 1:4); outside the timed region.
    for pol in ("mean", "gittins-static", "gittins"):
        o, lv, inf_n = simulator.policy_order(pol, mass, plen, store.bin_repr, tr.arrival, tr.output_len,
                                              bucket, noise=0.2)
        host_orders[pol + "+noise"] = (o.cpu().numpy(), lv, inf_n, pol == "gittins")
    # The same policies on the semantic-unaware predictor (Sec. 4.3: the
    # history records with the most similar input length), outside the timed
    # region. The stand-in data carry no relation between input and output
    # length, so its distributions are close to the store's overall one.
    len_index = sage.LengthIndex(dev(w.hist_prompt_len), spec.L_max)
    mass_len = torch.empty_like(mass)
    for s in range(0, R, chunk):
        e = min(R, s + chunk)
        sage.predict_by_length(plen[s:e], len_index, store.hist_len, spec.k, spec.tau, store.bin_edges,
                               out=tuple(t[:e - s] for t in pred_out) + (mass_len[s:e],))
    for pol in ("mean", "gittins-static", "gittins"):
        o, lv, inf_n = simulator.policy_order(pol, mass_len, plen, store.bin_repr, tr.arrival, tr.output_len,
                                              bucket)
        host_orders[pol + "+length"] = (o.cpu().numpy(), lv, inf_n, pol == "gittins")

    def replay(arrival, servers, rate_s):
        out = {}
        for pol, (o, lv, inf_n, refresh) in host_orders.items():
            t1 = time.perf_counter()
            finish, pre = sage.simulate(arrival, tr.prompt_len, tr.output_len, o, rate=rate_s,
                                        servers=servers, queue_cap=cap, bucket=bucket if refresh else 0,
                                        levels=lv, informed=inf_n)
            T = finish - arrival
            out[pol] = {"mean_ttlt_s": float(T.mean()), "p99_ttlt_s": float(np.percentile(T, 99)),
                        "preemptions": int(pre.sum()), "replay_ms": 1e3 * (time.perf_counter() - t1)}
        base = out["gittins"]["mean_ttlt_s"]
        for pol in out:
            out[pol]["gittins_reduction"] = 1.0 - base / out[pol]["mean_ttlt_s"]
        return out

    policies = replay(tr.arrival, nodes, rate)
    # the same requests on one server at 8 requests/s (arrival times stretched by the
    # number of servers; the queue orders do not depend on the arrival times)
    rate1 = simulator.rate_for_load(tr.prompt_len, tr.output_len, 8.0, 1, args.load)
    single = replay(tr.arrival * nodes, 1, rate1)

    k1_avg_s = k1_ms / n_launch / 1e3
    rows = R / n_launch * args.steps                 # queries per predict launch (chunked)
    flops = 2.0 * rows * spec.N * spec.d
    achieved = flops / k1_avg_s / 1e12
    line = {
        "metric": "scheduling decisions/sec (predict+cost+index+rank)",
        "value": R * args.steps / elapsed,
        "unit": "decisions/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": 1e3 * elapsed / args.steps,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": f"ttlt: {R}-request Poisson trace at 8 req/s x {nodes} servers over "
                               f"the mid store (N={spec.N} d={spec.d} k={spec.k} B={spec.B}), "
                               f"load {args.load}, <= {cap} queued, bucket {bucket}",
                   "R": R, "servers": nodes, "rps": rps, "load": args.load, "queue_cap": cap,
                   "bucket": bucket, "levels": L, "rate_cost_per_s": rate, "seed": [workloads.SEED_BASE, 2]},
        "policies": policies,
        "single_server": {"rps": 8.0, "rate_cost_per_s": rate1, "policies": single},
        "gpu_us_per_request": 1e6 * elapsed / args.steps / R,
        "roofline": {"bound": "mfma", "kernel": kernel_name(spec.k), "achieved": achieved,
                     "peak": MFMA_BF16_PEAK_TFLOPS, "unit": "TFLOP/s",
                     "frac": achieved / MFMA_BF16_PEAK_TFLOPS, "traffic": None,
                     "avg_launch_us": k1_avg_s * 1e6, "flops_per_launch": flops},
        "stages_us_per_step": {name: 1e3 * ms / args.steps for name, (n, ms) in stages.items()},
        "stage_rooflines": stage_rooflines({n: v for n, v in stages.items() if n != "index_scan"},
                                           rows, spec.d, spec.k, spec.B),
    }
    if not args.no_cpu_baseline:
        import copy
        ws = copy.copy(w)
        ws.queries, ws.prompt_len = tr.queries, tr.prompt_len
        ws.spec = copy.copy(spec)
        ws.spec.Q = R
        line["cpu_baseline"] = cpu_baseline(ws, args.cpu_seconds)
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
