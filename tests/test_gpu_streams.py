"""The binding on a side stream.  Outputs, workspaces and the zero-filled
value-gradient table that a call allocates belong to the stream it launches on
(the `stream` argument), so the whole path run on a side stream with nothing
passed in gives what it gives on the current stream: bitwise for the
deterministic kernels, within fp32 rounding for the atomic value gradient.
Between the side-stream calls the current stream allocates and fills memory
of its own, which must not land in a block the side stream still uses."""
import pytest
import torch

import paper_2412_09764_amd as pk
from paper_2412_09764_amd.inputs import WORKLOADS, gen_dy, gen_queries, gen_subkeys, gen_values

pytestmark = pytest.mark.gpu


def _path(q, K, V, dy, k, mode, stream=None, churn=None):
    outs = {}
    idx, w, score, _ = pk.mem_search(q, K, k, stream=stream)
    if churn:
        churn()
    y = pk.mem_bag_forward(V, idx.view(q.shape[0], -1), w.view(q.shape[0], -1), stream=stream)
    if churn:
        churn()
    gv, gw, gz = pk.mem_bag_backward(dy, V, idx, w, mode=mode, stream=stream)
    if churn:
        churn()
    gq, gK = pk.mem_search_backward(q, K, idx, gz, stream=stream)
    if churn:
        churn()
    outs.update(idx=idx, w=w, score=score, y=y, gv=gv, gw=gw, gz=gz, gq=gq, gK=gK)
    return outs


@pytest.mark.parametrize("mode", ["sorted", "atomic"])
def test_side_stream_matches_current_stream(gpu_lib, mode):
    dev = torch.device("cuda:0")
    wl = WORKLOADS["pk1m_d1024"]
    T = 2048
    q = gen_queries(wl, dev, T=T)
    K = gen_subkeys(wl, dev)
    V = gen_values(wl, dev)
    dy = gen_dy(wl, dev, T=T)
    ref = _path(q, K, V, dy, wl.k, mode)
    torch.cuda.synchronize()

    junk = []

    def churn():  # allocations and writes of the current stream
        t = torch.empty(64 << 20, dtype=torch.uint8, device=dev)
        t.fill_(0xAB)
        junk.append(t)
        if len(junk) > 4:
            junk.pop(0)

    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    got = _path(q, K, V, dy, wl.k, mode, stream=s, churn=churn)
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    exact = ["idx", "w", "score", "y", "gw", "gz", "gq", "gK"] + (["gv"] if mode == "sorted" else [])
    for name in exact:
        assert torch.equal(ref[name], got[name]), name
    if mode == "atomic":
        err = (ref["gv"] - got["gv"]).abs().max() / ref["gv"].abs().max()
        assert err <= 1e-5, err
