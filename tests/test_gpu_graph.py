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


def test_sink_step_replayed_from_a_hip_graph(gpu_lib):
    """The same with extra pairs and the sink pair: search_sink, bag forward
    and sorted backward over k + r + 1 slots, search_backward_sink (grad_q,
    grad_subkeys and grad_sink accumulate across replays)."""
    S, H, n, k, r, T, D = 128, 2, 64, 8, 4, 600, 128
    N = S * S + H
    dev = torch.device("cuda:0")
    g = torch.Generator().manual_seed(4)
    q = torch.randn((T, H, n), generator=g).to(torch.bfloat16).to(dev)
    K = (torch.randn((H, 2, S, n // 2), generator=g) / 8).to(torch.bfloat16).to(dev)
    ks = (torch.randn((H, n), generator=g) / 8).to(torch.bfloat16).to(dev)
    ex = torch.randint(0, S * S, (T, H, r), generator=g).to(dev)
    V = (torch.randn((N, D), generator=g) * 0.02).to(torch.bfloat16).to(dev)
    dy = torch.randn((T, D), generator=g).to(torch.bfloat16).to(dev)
    kk = k + r + 1
    idx = torch.empty((T, H, kk), dtype=torch.int64, device=dev)
    w = torch.empty((T, H, kk), dtype=torch.float32, device=dev)
    score = torch.empty_like(w)
    y = torch.empty((T, D), dtype=torch.bfloat16, device=dev)
    gv = torch.zeros((N, D), dtype=torch.float32, device=dev)
    gw = torch.empty_like(w)
    gz = torch.empty_like(w)
    gq = torch.empty((T, H, n), dtype=torch.float32, device=dev)
    gK = torch.zeros((H, 2, S, n // 2), dtype=torch.float32, device=dev)
    gS = torch.zeros((H, n), dtype=torch.float32, device=dev)
    ws_s = torch.empty(pk.mem_search_workspace_size(T, H, S, k), dtype=torch.uint8, device=dev)
    ws_b = torch.empty(pk.mem_bag_backward_workspace_size(T, H, kk, N, D, "sorted"),
                       dtype=torch.uint8, device=dev)
    ws_q = torch.empty(pk.load().mem_search_backward_sink_workspace_size(T, H, n, S, k + r),
                       dtype=torch.uint8, device=dev)

    def step(stream):
        pk.mem_search_sink(q, K, k, ks, S * S, ex, idx_out=idx, w_out=w, score_out=score,
                           workspace=ws_s, stream=stream)
        pk.mem_bag_forward(V, idx.view(T, -1), w.view(T, -1), y_out=y, stream=stream)
        pk.mem_bag_backward(dy, V, idx, w, grad_values=gv, grad_w=gw, grad_scores=gz, mode="sorted",
                            workspace=ws_b, stream=stream)
        pk.mem_search_backward_sink(q, K, idx, gz, ks, grad_q=gq, grad_subkeys=gK, grad_sink=gS,
                                    workspace=ws_q, stream=stream)

    bufs = (idx, w, score, y, gw, gz, gq, gv, gK, gS)
    ref = []
    st = torch.cuda.current_stream()
    for _ in range(3):
        step(st)
        torch.cuda.synchronize()
        ref.append([t.clone() for t in bufs])
    for t in (gv, gK, gS):
        t.zero_()
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
    assert float(gS.abs().sum()) == 0.0

    names = ("idx", "w", "score", "y", "grad_w", "grad_scores", "grad_q", "grad_values",
             "grad_subkeys", "grad_sink")
    for rep in range(3):
        graph.replay()
        torch.cuda.synchronize()
        for name, a, b in zip(names, bufs, ref[rep]):
            assert torch.equal(a, b), f"replay {rep}: {name} differs from the eager step"
        _ = (dy.float() * 2).sum().item()
