"""A whole scheduling decision (query ingest, predict, fused cost + index,
rank) enqueues kernels only: no allocation, copy, memset or synchronisation.
It can therefore be captured once in a HIP graph and replayed, as a serving
loop would. Each replay is checked bit for bit against the eager run, with
eager work between the replays that overwrites every output.
"""
import numpy as np
import pytest
import torch

from paper_2603_07917_amd import sage, workloads

pytestmark = pytest.mark.gpu

PANELS = 1


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


class Decision:
    """Resident inputs, preallocated outputs and workspaces of one decision."""

    def __init__(self, w):
        spec = w.spec
        self.Q, self.N, self.d, self.k, self.B = spec.Q, spec.N, spec.d, spec.k, spec.B
        self.tau = float(spec.tau)
        Q, d, k, B = self.Q, self.d, self.k, self.B
        self.hist = sage.ingest_bf16(dev(w.hist_emb), "panels")
        self.hist_len, self.edges, self.repr = dev(w.hist_len), dev(w.bin_edges), dev(w.bin_repr)
        self.queries, self.plen = dev(w.queries), dev(w.prompt_len)
        self.qb = torch.empty((d // 32, Q, 32), dtype=torch.bfloat16, device="cuda")
        self.out = [torch.empty((Q, k), dtype=torch.int32, device="cuda"),
                    torch.empty((Q, k), dtype=torch.float32, device="cuda"),
                    torch.empty((Q, B), dtype=torch.int32, device="cuda"),
                    torch.empty((Q, B), dtype=torch.float32, device="cuda"),
                    torch.empty(Q, dtype=torch.float32, device="cuda"),
                    torch.empty(Q, dtype=torch.int32, device="cuda")]
        self.ws = torch.empty(max(16, sage.predict_workspace_bytes(Q, self.N, d, k, B)), dtype=torch.uint8,
                              device="cuda")
        self.rws = torch.empty(max(16, sage.rank_workspace_bytes(Q)), dtype=torch.uint8, device="cuda")

    def step(self):
        lib = sage.load_library()
        s = torch.cuda.current_stream().cuda_stream        # the capturing stream inside a capture
        ids, sims, counts, mass, g, order = self.out
        sage._check(lib.sage_ingest_bf16_panels(self.queries.data_ptr(), self.Q, self.d, self.qb.data_ptr(), s))
        sage._check(lib.sage_predict_layout(self.qb.data_ptr(), PANELS, self.Q, self.hist.data_ptr(), PANELS,
                                            self.hist_len.data_ptr(), self.N, self.d, self.k, self.tau,
                                            self.edges.data_ptr(), self.B, ids.data_ptr(), sims.data_ptr(),
                                            counts.data_ptr(), mass.data_ptr(), self.ws.data_ptr(),
                                            self.ws.numel(), s))
        sage._check(lib.sage_index(mass.data_ptr(), None, self.plen.data_ptr(), self.repr.data_ptr(), self.Q,
                                   self.B, g.data_ptr(), None, s))
        sage._check(lib.sage_rank(g.data_ptr(), self.Q, order.data_ptr(), self.rws.data_ptr(), self.rws.numel(), s))

    def snapshot(self):
        torch.cuda.synchronize()
        return [t.cpu().numpy().copy() for t in self.out]


@pytest.mark.parametrize("Q,N,d,k,B", [
    (300, 40000, 64, 32, 64),       # filtered path with its threshold pre-pass; counting rank
    (8, 70000, 96, 128, 128),       # stream path
    (20000, 30000, 64, 16, 32),     # filtered path; the radix rank (more than 16,384 requests)
])
def test_decision_replays_in_a_hip_graph(Q, N, d, k, B):
    print(f"case Q={Q} N={N} d={d} k={k} B={B}", flush=True)
    w = workloads.small_predict(Q=Q, N=N, d=d, k=k, B=B, seed=Q + N + k, clusters=6)
    dec = Decision(w)
    dec.step()
    eager = dec.snapshot()

    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        dec.step()                                      # a run on the capture stream before capturing
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        dec.step()
    torch.cuda.synchronize()

    for r in range(4):
        for t in dec.out:                               # eager work between replays
            t.fill_(-3 - r)
        dec.ws.fill_(0xA5)
        torch.cuda.synchronize()
        graph.replay()
        got = dec.snapshot()
        for a, b in zip(eager, got):
            assert np.array_equal(a.view(np.uint8), b.view(np.uint8)), f"replay {r}"
        dec.step()                                      # and an eager decision in between
        for a, b in zip(eager, dec.snapshot()):
            assert np.array_equal(a.view(np.uint8), b.view(np.uint8)), f"eager after replay {r}"
