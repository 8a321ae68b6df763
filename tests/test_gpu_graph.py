"""A whole training step of the memory layer (search, bag forward, sorted bag
backward, search backward) captured once in a HIP graph and replayed: the
library allocates nothing, issues no memset and never waits on the host in
these calls, so the captured step must reproduce the eager step bit for bit
(the sorted backward and the search backward are deterministic).  Every
replay is checked against its own eager counterpart, with eager work and
synchronisations between the replays."""
import pytest
import torch

import paper_2412_09764_amd as pk
from tests.test_gpu_parity import int_tensor

pytestmark = pytest.mark.gpu


def test_step_replayed_from_a_hip_graph(gpu_lib):
    S, H, n, k, T, D = 256, 2, 64, 8, 300, 256
    N = S * S
    dev = torch.device("cuda:0")
    g = torch.Generator().manual_seed(3)
    q = (torch.randn((T, H, n), generator=g)).to(torch.bfloat16).to(dev)
    K = (torch.randn((H, 2, S, n // 2), generator=g) / 8).to(torch.bfloat16).to(dev)
    V = (torch.randn((N, D), generator=g) * 0.02).to(torch.bfloat16).to(dev)
    dy = torch.randn((T, D), generator=g).to(torch.bfloat16).to(dev)

    # every buffer the step touches, allocated before capture
    idx = torch.empty((T, H, k), dtype=torch.int64, device=dev)
    w = torch.empty((T, H, k), dtype=torch.float32, device=dev)
    score = torch.empty_like(w)
    y = torch.empty((T, D), dtype=torch.bfloat16, device=dev)
    gv = torch.zeros((N, D), dtype=torch.float32, device=dev)
    gw = torch.empty_like(w)
    gz = torch.empty_like(w)
    gq = torch.empty((T, H, n), dtype=torch.float32, device=dev)
    gK = torch.zeros((H, 2, S, n // 2), dtype=torch.float32, device=dev)
    ws_s = torch.empty(pk.mem_search_workspace_size(T, H, S, k), dtype=torch.uint8, device=dev)
    ws_b = torch.empty(pk.mem_bag_backward_workspace_size(T, H, k, N, D, "sorted"),
                       dtype=torch.uint8, device=dev)
    ws_q = torch.empty(pk.load().mem_search_backward_workspace_size(T, H, S, k), dtype=torch.uint8,
                       device=dev)

    def step(stream):
        pk.mem_search(q, K, k, idx_out=idx, w_out=w, score_out=score, workspace=ws_s, stream=stream)
        pk.mem_bag_forward(V, idx.view(T, -1), w.view(T, -1), y_out=y, stream=stream)
        pk.mem_bag_backward(dy, V, idx, w, grad_values=gv, grad_w=gw, grad_scores=gz, mode="sorted",
                            workspace=ws_b, stream=stream)
        pk.mem_search_backward(q, K, idx, gz, grad_q=gq, grad_subkeys=gK, workspace=ws_q,
                               stream=stream)

    # eager reference: three steps, state after each (gradients accumulate)
    ref = []
    st = torch.cuda.current_stream()
    for _ in range(3):
        step(st)
        torch.cuda.synchronize()
        ref.append([t.clone() for t in (idx, w, score, y, gw, gz, gq, gv, gK)])
    gv.zero_()
    gK.zero_()
    for t in (idx, w, score, y, gw, gz, gq):
        t.fill_(0)
    torch.cuda.synchronize()

    graph = torch.cuda.CUDAGraph()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        with torch.cuda.graph(graph, stream=side):
            step(side)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    # capture does not execute: gradients are still zero
    assert float(gv.abs().sum()) == 0.0 and float(gK.abs().sum()) == 0.0

    names = ("idx", "w", "score", "y", "grad_w", "grad_scores", "grad_q", "grad_values",
             "grad_subkeys")
    for r in range(3):
        graph.replay()
        torch.cuda.synchronize()
        got = (idx, w, score, y, gw, gz, gq, gv, gK)
        for name, a, b in zip(names, got, ref[r]):
            assert torch.equal(a, b), f"replay {r}: {name} differs from the eager step"
        # eager work between replays (must not disturb the graph's buffers)
        _ = (dy.float() * 2).sum().item()
