"""The library's calls inside a captured HIP graph (torch.cuda.CUDAGraph):
every replay equals the eager call bitwise, also with other eager library
work on the same buffers shapes between replays (the library records no
memset nodes and allocates nothing; its counters are cleared by its own
fill kernels, so replays after the first are as correct as the first)."""
import numpy as np
import pytest

pytestmark = pytest.mark.gpu


def _setup(M, N, D, C, seed):
    import torch
    rng = np.random.default_rng(seed)
    dev = torch.device("cuda:0")
    q = torch.from_numpy(rng.standard_normal((M, D)).astype(np.float16)).to(dev)
    k = torch.from_numpy(rng.standard_normal((N, D)).astype(np.float16)).to(dev)
    v = torch.from_numpy(rng.standard_normal((N, C)).astype(np.float32)).to(dev)
    g = torch.from_numpy(rng.standard_normal((M, C)).astype(np.float32)).to(dev)
    return q, k, v, g


@pytest.mark.parametrize("M,N,D,C,mode", [(4096, 4096, 16, 1, "fwd"), (3000, 5000, 64, 1, "fwd_bwd"),
                                          (1000, 1500, 40, 12, "fwd_bwd"), (700, 1200, 256, 16, "fwd_bwd")])
def test_graph_replays_match_eager(M, N, D, C, mode):
    import torch
    from paper_2609_04910_amd import gauss_sum as gs

    q, k, v, g = _setup(M, N, D, C, seed=M + D)
    tau = 1.0 / D
    want = (True, True, True)
    if mode == "fwd":
        ws = torch.empty(max(gs.gauss_sum_fwd_workspace_size(M, N, D, C, gs.GS_F16, gs.GS_F32), 1),
                         dtype=torch.uint8, device="cuda")
    else:
        ws = torch.empty(max(gs.gauss_sum_fwd_bwd_workspace_size(M, N, D, C, gs.GS_F16, gs.GS_F32, *want), 1),
                         dtype=torch.uint8, device="cuda")
    outs = {"s": torch.empty((M, C), dtype=torch.float32, device="cuda")}

    def call(stream):
        if mode == "fwd":
            gs.gauss_sum_fwd(q, k, v, tau, out=outs["s"], workspace=ws, stream=stream)
            return (outs["s"],)
        _, dq, dk, dv = gs.gauss_sum_fwd_bwd(q, k, v, tau, g, want=want, out=outs["s"], workspace=ws,
                                             stream=stream)
        return outs["s"], dq, dk, dv

    eager = [t.clone() for t in call(torch.cuda.current_stream())]
    torch.cuda.synchronize()

    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        call(side)  # warm-up on the capture stream's side, as torch recommends
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        captured = call(torch.cuda.current_stream())
    torch.cuda.synchronize()

    q2, k2, v2, g2 = _setup(M, N, D, C, seed=M + D + 1)
    for rep in range(3):
        for t in captured:
            t.fill_(float("nan"))
        graph.replay()
        torch.cuda.synchronize()
        for name, got, ref in zip(("s", "dq", "dk", "dv"), captured, eager):
            assert torch.equal(got, ref), "replay %d: %s differs from the eager call" % (rep, name)
        # other eager work with the library (other inputs, own workspace) in between
        if mode == "fwd":
            gs.gauss_sum_fwd(q2, k2, v2, tau)
        else:
            gs.gauss_sum_fwd_bwd(q2, k2, v2, tau, g2, want=want)
        torch.cuda.synchronize()
