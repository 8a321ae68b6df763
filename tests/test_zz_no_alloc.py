"""mem_search_noalloc: the search with its workspace in the library's static
device scratch array, for callers that cannot allocate.  Through the C ABI it
must give bitwise what mem_search gives with a caller workspace (the same
kernels on the same inputs), call after call, including a smaller call after
a larger one (the array keeps the previous call's contents), and, on integer
inputs, the oracle's selection exactly."""

import numpy as np
import pytest
import torch

import oracle
import paper_2412_09764_amd as pk
from paper_2412_09764_amd.inputs import WORKLOADS, gen_queries, gen_subkeys


def _searches(L, q, K, k):
    """(mem_search with a workspace, mem_search_noalloc) outputs as host tensors."""
    T, H, n = q.shape
    S = K.shape[2]
    dt = pk.BF16 if q.dtype == torch.bfloat16 else pk.F32
    st = torch.cuda.current_stream().cuda_stream
    res = []
    for noalloc in (False, True):
        idx = torch.full((T, H, k), -7, dtype=torch.int64, device=q.device)
        w = torch.full((T, H, k), float("nan"), dtype=torch.float32, device=q.device)
        sc = torch.full((T, H, k), float("nan"), dtype=torch.float32, device=q.device)
        hi = torch.full((T, H, 2, k), -7, dtype=torch.int32, device=q.device)
        if noalloc:
            rc = L.mem_search_noalloc(q.data_ptr(), dt, K.data_ptr(), dt, T, H, n, S, k,
                                      idx.data_ptr(), w.data_ptr(), sc.data_ptr(), hi.data_ptr(), st)
        else:
            ws = torch.empty(L.mem_search_workspace_size(T, H, S, k), dtype=torch.uint8,
                             device=q.device)
            rc = L.mem_search(q.data_ptr(), dt, K.data_ptr(), dt, T, H, n, S, k, idx.data_ptr(),
                              w.data_ptr(), sc.data_ptr(), hi.data_ptr(), ws.data_ptr(), ws.numel(),
                              st)
        assert rc == 0, L.mem_last_error().decode()
        torch.cuda.synchronize()
        res.append((idx.cpu(), w.cpu(), sc.cpu(), hi.cpu()))
    return res


def _same(a, b):
    for x, y, name in zip(a, b, ("idx", "w", "score", "half_idx")):
        assert torch.equal(x.view(torch.int32) if x.dtype == torch.float32 else x,
                           y.view(torch.int32) if y.dtype == torch.float32 else y), name


@pytest.mark.gpu
def test_noalloc_matches_workspace_search_twice(gpu_lib):
    L = gpu_lib.load()
    dev = torch.device("cuda:0")
    wl = WORKLOADS["pk1m_d1024"]  # S = 1024, H = 4, n = 512, k = 32, bf16
    K = gen_subkeys(wl, dev)
    # first call: 4096 tokens (about 76 MB of the 128 MiB scratch), Gaussian queries
    T1 = 4096
    assert pk.mem_search_workspace_size(T1, wl.H, wl.S, wl.k) <= pk.NOALLOC_SCRATCH_BYTES
    q1 = gen_queries(wl, dev, T=T1)
    ref1, got1 = _searches(L, q1, K, wl.k)
    _same(ref1, got1)
    # second call, smaller and ragged (300 tokens), integer inputs: also the oracle's
    Ki = gen_subkeys(wl, dev, integer=True)
    q2 = gen_queries(wl, dev, integer=True, T=300)
    ref2, got2 = _searches(L, q2, Ki, wl.k)
    _same(ref2, got2)
    s = oracle.search(q2.cpu().double().numpy(), Ki.cpu().double().numpy(), wl.k)
    assert np.array_equal(got2[0].numpy(), s["idx"])
    rel = np.abs(got2[1].double().numpy() - s["w"]).max() / np.abs(s["w"]).max()
    assert rel <= 1e-5, rel


@pytest.mark.gpu
def test_noalloc_fp32_small_after_large(gpu_lib):
    L = gpu_lib.load()
    dev = torch.device("cuda:0")
    wl = WORKLOADS["pk4k_d64_f32"]  # S = 64, H = 1, n = 64, k = 8, fp32
    K = gen_subkeys(wl, dev, integer=True)
    for T in (wl.T, 37):
        q = gen_queries(wl, dev, integer=True, T=T)
        ref, got = _searches(L, q, K, wl.k)
        _same(ref, got)
        s = oracle.search(q.cpu().double().numpy(), K.cpu().double().numpy(), wl.k)
        assert np.array_equal(got[0].numpy(), s["idx"])


@pytest.mark.gpu
def test_noalloc_binding_on_side_stream(gpu_lib):
    """The Python wrapper on a side stream gives what mem_search gives."""
    dev = torch.device("cuda:0")
    wl = WORKLOADS["pk1m_d1024"]
    K = gen_subkeys(wl, dev)
    q = gen_queries(wl, dev, T=1000)
    ref = pk.mem_search(q, K, wl.k, want_half=True)
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        got = pk.mem_search_noalloc(q, K, wl.k, want_half=True, stream=s)
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    for a, b in zip(ref, got):
        assert torch.equal(a, b)


def test_noalloc_rejects_beyond_scratch():
    """Checked on the host before any device call (fake, aligned pointers)."""
    L = pk.load()
    wl = WORKLOADS["pk4m_d2048"]
    T = wl.T  # 32768 tokens x 4 heads: about 340 MB of workspace
    assert pk.mem_search_workspace_size(T, wl.H, wl.S, wl.k) > pk.NOALLOC_SCRATCH_BYTES
    fake = 0x10000
    rc = L.mem_search_noalloc(fake, pk.BF16, fake, pk.BF16, T, wl.H, wl.n, wl.S, wl.k, fake, fake,
                              None, None, None)
    assert rc == -2
    assert "scratch" in L.mem_last_error().decode()
