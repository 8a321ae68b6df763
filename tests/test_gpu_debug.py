"""PKMEM_DEBUG=1: the calls that index with idx check on the device that
every index is in range first and fail with PKMEM_ERR_INVALID if one is not
(no kernel reads out of range).  Also: the search is deterministic run to run."""
import pytest
import torch

import paper_2412_09764_amd as pk
from tests.test_gpu_parity import normal_tensor

pytestmark = pytest.mark.gpu

INVALID = -1


def _bag_case():
    g = torch.Generator().manual_seed(111)
    N, D, T, H, k = 500, 64, 20, 2, 4
    V = (torch.randn((N, D), generator=g) * 0.1).to(torch.bfloat16).cuda()
    idx = torch.randint(0, N, (T, H, k), generator=g).cuda()
    w = torch.rand((T, H, k), generator=g).cuda()
    dy = torch.randn((T, D), generator=g).to(torch.bfloat16).cuda()
    return V, idx, w, dy


def test_debug_checks_reject_out_of_range_indices(gpu_lib, monkeypatch):
    V, idx, w, dy = _bag_case()
    T = idx.shape[0]
    N = V.shape[0]
    ref = pk.mem_bag_forward(V, idx.view(T, -1), w.view(T, -1))
    monkeypatch.setenv("PKMEM_DEBUG", "1")
    # in range: same result as without the check
    assert torch.equal(pk.mem_bag_forward(V, idx.view(T, -1), w.view(T, -1)), ref)
    bad = idx.clone()
    bad[3, 1, 2] = N
    with pytest.raises(pk.PkmemError) as e:
        pk.mem_bag_forward(V, bad.view(T, -1), w.view(T, -1))
    assert e.value.code == INVALID and "PKMEM_DEBUG" in str(e.value)
    bad[3, 1, 2] = -1
    for mode in ("sorted", "atomic"):
        with pytest.raises(pk.PkmemError) as e:
            pk.mem_bag_backward(dy, V, bad, w, mode=mode)
        assert e.value.code == INVALID
    with pytest.raises(pk.PkmemError):
        pk.mem_bag_forward_gated(V, bad.view(T, -1), w.view(T, -1), dy)
    S, H, n, k = 16, 2, 32, 4
    q = normal_tensor((T, H, n), 112, torch.bfloat16).cuda()
    K = normal_tensor((H, 2, S, n // 2), 113, torch.bfloat16).cuda()
    sidx, _, _, _ = pk.mem_search(q, K, k)
    sidx[0, 0, 0] = S * S
    with pytest.raises(pk.PkmemError):
        pk.mem_search_backward(q, K, sidx, torch.ones((T, H, k), device="cuda"))
    monkeypatch.delenv("PKMEM_DEBUG")
    torch.cuda.synchronize()


def test_debug_checks_with_a_sink_slot(gpu_lib, monkeypatch):
    """The sink's slot (index >= S*S by construction) passes the check of the
    sink search backward, which covers the product-key slots only; a bad
    product-key index or a bad extra index is rejected."""
    T, S, H, n, k = 20, 16, 2, 32, 4
    q = normal_tensor((T, H, n), 116, torch.bfloat16).cuda()
    K = normal_tensor((H, 2, S, n // 2), 117, torch.bfloat16).cuda()
    ks = normal_tensor((H, n), 118, torch.bfloat16).cuda()
    idx, w, _, _ = pk.mem_search_sink(q, K, k, ks, S * S)
    gz = torch.ones((T, H, k + 1), device="cuda")
    ref = pk.mem_search_backward_sink(q, K, idx, gz, ks)
    monkeypatch.setenv("PKMEM_DEBUG", "1")
    got = pk.mem_search_backward_sink(q, K, idx, gz, ks)
    for a, b in zip(ref, got):
        assert torch.equal(a, b)
    bad = idx.clone()
    bad[5, 1, k - 1] = -3
    with pytest.raises(pk.PkmemError) as e:
        pk.mem_search_backward_sink(q, K, bad, gz, ks)
    assert e.value.code == INVALID
    ex = torch.zeros((T, H, 2), dtype=torch.int64, device="cuda")
    ex[7, 0, 1] = S * S
    with pytest.raises(pk.PkmemError) as e:
        pk.mem_search_sink(q, K, k, ks, S * S, ex)
    assert e.value.code == INVALID
    monkeypatch.delenv("PKMEM_DEBUG")
    torch.cuda.synchronize()


def test_search_is_deterministic_run_to_run(gpu_lib):
    q = normal_tensor((700, 4, 512), 114, torch.bfloat16).cuda()
    K = normal_tensor((4, 2, 2048, 256), 115, torch.bfloat16, std=1 / 256).cuda()
    a = pk.mem_search(q, K, 32)
    b = pk.mem_search(q, K, 32)
    torch.cuda.synchronize()
    for x, y in zip(a[:3], b[:3]):
        assert torch.equal(x, y)
